// Attention backward with the GProj correction on gfx950 bf16 MFMA
// (Algorithm 1; appendix "Implemented Arithmetic and Rounding", eqs.
// gproj-row-mass, gproj-accumulators, gproj-query-implemented,
// gproj-key-implemented).
//
// Schedule (deterministic, no atomics).  Algorithm 1 accumulates dQ and B = rK
// with atomic adds from a key-major loop and then needs a second key-major pass
// for dK, because lambda_i = rho_i / m_i is known only after row i has seen
// every key.  Here the same arithmetic is split by ownership instead:
//   1. bwd_pre   : D_i = rowsum(dO_i * O_i) in FP32.
//   2. bwd_dq    : query-major.  A workgroup owns 64 query rows and streams the
//                  key tiles, so A = tK, B = rK, rho and m stay in registers; at
//                  the end it forms lambda = rho/m once and writes
//                  dQ = BF16(fl32[alpha (A - lambda B)]) and lambda.
//   3. bwd_dkdv  : key-major.  A workgroup owns 64 keys and streams the query
//                  tiles; with lambda already known it accumulates dV = r^T dO,
//                  dK^acc = t^T Q and C = r^T z (z = BF16(lambda q), formed while
//                  the query tile is staged) and writes
//                  dK = BF16(fl32[alpha (dK^acc - C)]).
// Both passes rebuild P, r and t with identical instructions, so the r and t
// of the key pass equal those of the query pass bitwise, and lambda is divided
// once.  gproj_q runs the plain key-major pass; gproj runs the plain
// query-major pass plus the correction.  FP32 accumulators, BF16 operands and
// the cast points are those of the paper; only where lambda becomes available
// differs.
//
// MFMA layouts (v_mfma_f32_16x16x32_bf16, wave64): an A operand holds one row
// per lane (row = lane & 15) and 8 values along k; a B operand holds one column
// per lane; the 16x16 accumulator holds column lane & 15 and rows
// 4*(lane >> 4) + i.  Computing S^T = K Q^T (query-major) or S = Q K^T
// (key-major) leaves each lane with the probabilities of its own column in
// exactly the k-layout the next product needs, so P, r and t never pass
// through LDS.
#include "gpa_device.h"
#include "gpa_launch.h"

namespace gpa {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---------------------------------------------------------------- preprocess
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const uint16_t* __restrict__ O,
                                                      const uint16_t* __restrict__ dO,
                                                      float* __restrict__ Drow, int rows) {
    constexpr int TPR = D / 8;  // lanes per row, 8 elements each
    const int gid = blockIdx.x * 256 + threadIdx.x;
    const int row = gid / TPR;
    const int part = gid - row * TPR;
    float acc = 0.f;
    if (row < rows) {
        const u32x4 o = *reinterpret_cast<const u32x4*>(O + (size_t)row * D + part * 8);
        const u32x4 u = *reinterpret_cast<const u32x4*>(dO + (size_t)row * D + part * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            // BF16 x BF16 products are exact in FP32.
            acc += lo_bf16(u[e]) * lo_bf16(o[e]);
            acc += hi_bf16(u[e]) * hi_bf16(o[e]);
        }
    }
#pragma unroll
    for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (row < rows && part == 0) Drow[row] = acc;
}

// --------------------------------------------------------- query-major pass
template <int D, bool GPROJ>
__global__ __launch_bounds__(kThreads) void bwd_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow, uint16_t* __restrict__ dQ,
    float* __restrict__ rho_out, float* __restrict__ m_out, float* __restrict__ lam_out,
    int BH, int N, int causal, float scale) {
    constexpr int RP = Pitch<D>::row;
    constexpr int TP = Pitch<D>::tr;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kTile * RP];  // K row-major
    __shared__ __attribute__((aligned(16))) uint16_t Vs[kTile * RP];  // V row-major
    __shared__ __attribute__((aligned(16))) uint16_t Kt[D * TP];      // K transposed

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + wave * 16 + c16;
    const bool qok = qrow < N;
    const size_t ridx = (size_t)bh * N + qrow;

    bf16x8 qf[D / 32], uf[D / 32];
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
        u32x4 wq = {0u, 0u, 0u, 0u}, wu = {0u, 0u, 0u, 0u};
        if (qok) {
            wq = *reinterpret_cast<const u32x4*>(Q + hoff + (size_t)qrow * D + kc * 32 + 8 * g);
            wu = *reinterpret_cast<const u32x4*>(dO + hoff + (size_t)qrow * D + kc * 32 + 8 * g);
        }
        qf[kc] = __builtin_bit_cast(bf16x8, wq);
        uf[kc] = __builtin_bit_cast(bf16x8, wu);
    }
    const float c = scale * kLog2e;
    const float lse2 = qok ? LSE[ridx] * kLog2e : 0.f;
    const float Di = qok ? Drow[ridx] : 0.f;

    f32x4 accA[D / 16], accB[GPROJ ? D / 16 : 1];
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) accA[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mb = 0; mb < (GPROJ ? D / 16 : 1); ++mb) accB[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float rho = 0.f, msum = 0.f;

    const int nkv = causal ? min(T, tile + 1) : T;
    for (int kt = 0; kt < nkv; ++kt) {
        const int k0 = kt * kTile;
        __syncthreads();
        for (int ch = tid; ch < kTile * D / 8; ch += kThreads) {
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            const int row = k0 + r;
            u32x4 kw = {0u, 0u, 0u, 0u}, vw = {0u, 0u, 0u, 0u};
            if (row < N) {
                kw = *reinterpret_cast<const u32x4*>(K + hoff + (size_t)row * D + cc);
                vw = *reinterpret_cast<const u32x4*>(V + hoff + (size_t)row * D + cc);
            }
            *reinterpret_cast<u32x4*>(Ks + r * RP + cc) = kw;
            *reinterpret_cast<u32x4*>(Vs + r * RP + cc) = vw;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                Kt[(cc + 2 * e) * TP + r] = (uint16_t)(kw[e] & 0xFFFFu);
                Kt[(cc + 2 * e + 1) * TP + r] = (uint16_t)(kw[e] >> 16);
            }
        }
        __syncthreads();

        // S^T = K Q^T and dP^T = V dO^T: lane holds keys 4g+i of each 16-key
        // block for its own query.
        f32x4 s[4], dp[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
            dp[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < D / 32; ++kc) {
                s[kb] = mfma_16x16x32(ld_b128(Ks + (kb * 16 + c16) * RP + kc * 32 + 8 * g), qf[kc],
                                      s[kb]);
                dp[kb] = mfma_16x16x32(ld_b128(Vs + (kb * 16 + c16) * RP + kc * 32 + 8 * g),
                                       uf[kc], dp[kb]);
            }
        }
        bf16x8 tf[2], rf[2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = k0 + kb * 16 + 4 * g + i;
                const bool ok = qok && key < N && (!causal || key <= qrow);
                const float P = ok ? fexp2(fmaf(s[kb][i], c, -lse2)) : 0.f;
                const __bf16 rb = to_bf16(P);
                const __bf16 tb = to_bf16(P * (dp[kb][i] - Di));
                if (GPROJ) {
                    rho += bf16_to_f32(tb);
                    msum += bf16_to_f32(rb);
                }
                tf[kb >> 1][(kb & 1) * 4 + i] = tb;
                rf[kb >> 1][(kb & 1) * 4 + i] = rb;
            }
        // A^T[d][query] += K^T[d][key] t^T[key][query]  (and B^T with r).
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb)
#pragma unroll
            for (int kc2 = 0; kc2 < 2; ++kc2) {
                const uint16_t* a = Kt + (mb * 16 + c16) * TP + kc2 * 32 + 4 * g;
                const bf16x8 ka = ld_b64x2(a, a + 16);
                accA[mb] = mfma_16x16x32(ka, tf[kc2], accA[mb]);
                if (GPROJ) accB[mb] = mfma_16x16x32(ka, rf[kc2], accB[mb]);
            }
    }

    float lam = 0.f;
    if (GPROJ) {
        rho = xor_sum(rho);
        msum = xor_sum(msum);
        lam = (msum != 0.f) ? rho / msum : 0.f;  // one IEEE FP32 division
    }
    if (qok) {
        uint16_t* drow = dQ + hoff + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb) {
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                if (GPROJ) {
                    const float corr = lam * accB[mb][i];
                    const float diff = accA[mb][i] - corr;
                    v[i] = scale * diff;
                } else {
                    v[i] = scale * accA[mb][i];
                }
            }
            st_bf16x4(drow + mb * 16 + 4 * g, v[0], v[1], v[2], v[3]);
        }
        if (g == 0) {
            rho_out[ridx] = GPROJ ? rho : 0.f;
            m_out[ridx] = GPROJ ? msum : 0.f;
            lam_out[ridx] = lam;
        }
    }
}

// ----------------------------------------------------------- key-major pass
template <int D, bool GPROJ>
__global__ __launch_bounds__(kThreads) void bwd_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow,
    const float* __restrict__ lam, uint16_t* __restrict__ dK, uint16_t* __restrict__ dV,
    int BH, int N, int causal, float scale) {
    constexpr int RP = Pitch<D>::row;
    constexpr int TP = Pitch<D>::tr;
    __shared__ __attribute__((aligned(16))) uint16_t Qs[kTile * RP];   // Q row-major
    __shared__ __attribute__((aligned(16))) uint16_t Us[kTile * RP];   // dO row-major
    __shared__ __attribute__((aligned(16))) uint16_t Qt[D * TP];       // Q transposed
    __shared__ __attribute__((aligned(16))) uint16_t Ut[D * TP];       // dO transposed
    __shared__ __attribute__((aligned(16))) uint16_t Zt[GPROJ ? D * TP : 8];  // BF16(lambda q)^T
    __shared__ float lse2s[kTile];
    __shared__ float Ds[kTile];

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, false, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int krow = tile * kTile + wave * 16 + c16;
    const bool kok = krow < N;

    // K^T and V^T as B operands: column = this lane's key, k = d.
    bf16x8 kf[D / 32], vf[D / 32];
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
        u32x4 wk = {0u, 0u, 0u, 0u}, wv = {0u, 0u, 0u, 0u};
        if (kok) {
            wk = *reinterpret_cast<const u32x4*>(K + hoff + (size_t)krow * D + kc * 32 + 8 * g);
            wv = *reinterpret_cast<const u32x4*>(V + hoff + (size_t)krow * D + kc * 32 + 8 * g);
        }
        kf[kc] = __builtin_bit_cast(bf16x8, wk);
        vf[kc] = __builtin_bit_cast(bf16x8, wv);
    }
    const float c = scale * kLog2e;

    f32x4 accV[D / 16], accK[D / 16], accC[GPROJ ? D / 16 : 1];
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) {
        accV[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
        accK[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int mb = 0; mb < (GPROJ ? D / 16 : 1); ++mb) accC[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int qt0 = causal ? tile : 0;
    for (int qt = qt0; qt < T; ++qt) {
        const int q0 = qt * kTile;
        __syncthreads();
        for (int ch = tid; ch < kTile * D / 8; ch += kThreads) {
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            const int row = q0 + r;
            u32x4 qw = {0u, 0u, 0u, 0u}, uw = {0u, 0u, 0u, 0u};
            float lr = 0.f;
            if (row < N) {
                qw = *reinterpret_cast<const u32x4*>(Q + hoff + (size_t)row * D + cc);
                uw = *reinterpret_cast<const u32x4*>(dO + hoff + (size_t)row * D + cc);
                if (GPROJ) lr = lam[(size_t)bh * N + row];
            }
            *reinterpret_cast<u32x4*>(Qs + r * RP + cc) = qw;
            *reinterpret_cast<u32x4*>(Us + r * RP + cc) = uw;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                Qt[(cc + 2 * e) * TP + r] = (uint16_t)(qw[e] & 0xFFFFu);
                Qt[(cc + 2 * e + 1) * TP + r] = (uint16_t)(qw[e] >> 16);
                Ut[(cc + 2 * e) * TP + r] = (uint16_t)(uw[e] & 0xFFFFu);
                Ut[(cc + 2 * e + 1) * TP + r] = (uint16_t)(uw[e] >> 16);
                if (GPROJ) {
                    // z = BF16(fl32(lambda q))
                    Zt[(cc + 2 * e) * TP + r] = bf16_bits(lr * lo_bf16(qw[e]));
                    Zt[(cc + 2 * e + 1) * TP + r] = bf16_bits(lr * hi_bf16(qw[e]));
                }
            }
        }
        if (tid < kTile) {
            const int row = q0 + tid;
            const size_t ri = (size_t)bh * N + row;
            lse2s[tid] = row < N ? LSE[ri] * kLog2e : 0.f;
            Ds[tid] = row < N ? Drow[ri] : 0.f;
        }
        __syncthreads();

        // S = Q K^T and dP = dO V^T: lane holds queries 4g+i of each 16-query
        // block for its own key.
        f32x4 s[4], dp[4];
#pragma unroll
        for (int mq = 0; mq < 4; ++mq) {
            s[mq] = f32x4{0.f, 0.f, 0.f, 0.f};
            dp[mq] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < D / 32; ++kc) {
                s[mq] = mfma_16x16x32(ld_b128(Qs + (mq * 16 + c16) * RP + kc * 32 + 8 * g), kf[kc],
                                      s[mq]);
                dp[mq] = mfma_16x16x32(ld_b128(Us + (mq * 16 + c16) * RP + kc * 32 + 8 * g),
                                       vf[kc], dp[mq]);
            }
        }
        bf16x8 tf[2], rf[2];
#pragma unroll
        for (int mq = 0; mq < 4; ++mq)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ql = mq * 16 + 4 * g + i;
                const int query = q0 + ql;
                const bool ok = kok && query < N && (!causal || krow <= query);
                const float P = ok ? fexp2(fmaf(s[mq][i], c, -lse2s[ql])) : 0.f;
                tf[mq >> 1][(mq & 1) * 4 + i] = to_bf16(P * (dp[mq][i] - Ds[ql]));
                rf[mq >> 1][(mq & 1) * 4 + i] = to_bf16(P);
            }
        // dV^T[dv][key] += dO^T r ; dK^T += Q^T t ; C^T += Z^T r.
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb)
#pragma unroll
            for (int kc2 = 0; kc2 < 2; ++kc2) {
                const int off = (mb * 16 + c16) * TP + kc2 * 32 + 4 * g;
                accV[mb] = mfma_16x16x32(ld_b64x2(Ut + off, Ut + off + 16), rf[kc2], accV[mb]);
                accK[mb] = mfma_16x16x32(ld_b64x2(Qt + off, Qt + off + 16), tf[kc2], accK[mb]);
                if (GPROJ)
                    accC[mb] = mfma_16x16x32(ld_b64x2(Zt + off, Zt + off + 16), rf[kc2], accC[mb]);
            }
    }

    if (kok) {
        uint16_t* vrow = dV + hoff + (size_t)krow * D;
        uint16_t* krw = dK + hoff + (size_t)krow * D;
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb) {
            st_bf16x4(vrow + mb * 16 + 4 * g, accV[mb][0], accV[mb][1], accV[mb][2], accV[mb][3]);
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                if (GPROJ) {
                    const float diff = accK[mb][i] - accC[mb][i];
                    v[i] = scale * diff;
                } else {
                    v[i] = scale * accK[mb][i];
                }
            }
            st_bf16x4(krw + mb * 16 + 4 * g, v[0], v[1], v[2], v[3]);
        }
    }
}

}  // namespace

hipError_t launch_bwd_pre(const uint16_t* O, const uint16_t* dO, float* Drow, const Shape& s,
                          hipStream_t st) {
    const long rows = (long)s.BH * s.N;
    const int tpr = s.d / 8;
    const unsigned blocks = (unsigned)((rows * tpr + 255) / 256);
    if (s.d == 64)
        bwd_pre_kernel<64><<<blocks, 256, 0, st>>>(O, dO, Drow, (int)rows);
    else
        bwd_pre_kernel<128><<<blocks, 256, 0, st>>>(O, dO, Drow, (int)rows);
    return hipGetLastError();
}

hipError_t launch_bwd_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, const float* LSE, const float* Drow, uint16_t* dQ,
                         float* rho, float* msum, float* lambda, int mode, const Shape& s,
                         hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    const bool gp = mode != 0;
#define GPA_DQ(DD, GP)                                                                       \
    bwd_dq_kernel<DD, GP><<<grid, block, 0, st>>>(Q, K, V, dO, LSE, Drow, dQ, rho, msum, lambda, \
                                                  s.BH, s.N, s.causal, s.scale)
    if (s.d == 64) {
        if (gp) GPA_DQ(64, true); else GPA_DQ(64, false);
    } else {
        if (gp) GPA_DQ(128, true); else GPA_DQ(128, false);
    }
#undef GPA_DQ
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* LSE, const float* Drow,
                           const float* lambda, uint16_t* dK, uint16_t* dV, int mode,
                           const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    const bool gp = mode == 2;
#define GPA_DKDV(DD, GP)                                                                  \
    bwd_dkdv_kernel<DD, GP><<<grid, block, 0, st>>>(Q, K, V, dO, LSE, Drow, lambda, dK, dV, \
                                                    s.BH, s.N, s.causal, s.scale)
    if (s.d == 64) {
        if (gp) GPA_DKDV(64, true); else GPA_DKDV(64, false);
    } else {
        if (gp) GPA_DKDV(128, true); else GPA_DKDV(128, false);
    }
#undef GPA_DKDV
    return hipGetLastError();
}

}  // namespace gpa
