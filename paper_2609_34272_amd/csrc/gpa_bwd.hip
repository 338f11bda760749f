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
// through LDS.  The other operand of that product is read transposed from the
// row-major LDS tile with the LDS transpose load (ds_read_b64_tr_b16), so every
// tile is staged once, row-major, with 16-byte writes.
#include "gpa_device.h"
#include "gpa_launch.h"

namespace gpa {
namespace {


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
// P, r, t for one key tile of the query-major pass: lane holds keys 4g+i of
// each 16-key block for its query.  MASK applies causal and tail masks (only
// diagonal and tail tiles need them).
template <bool MASK>
__device__ __forceinline__ void dq_probs(const f32x4 (&s)[4], const f32x4 (&dp)[4], float c,
                                         float lse2, float Di, int k0, int g, int qrow, bool qok,
                                         int N, int causal, bf16x8 (&tf)[2], bf16x8 (&rf)[2]) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float P = fexp2(fmaf(s[kb][i], c, -lse2));
            if constexpr (MASK) {
                const int key = k0 + kb * 16 + 4 * g + i;
                const bool ok = qok && key < N && (!causal || key <= qrow);
                P = ok ? P : 0.f;
            }
            tf[kb >> 1][(kb & 1) * 4 + i] = to_bf16(P * (dp[kb][i] - Di));
            rf[kb >> 1][(kb & 1) * 4 + i] = to_bf16(P);
        }
}

template <int D, bool GPROJ>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow, uint16_t* __restrict__ dQ,
    float* __restrict__ rho_out, float* __restrict__ m_out, float* __restrict__ lam_out,
    int BH, int N, int causal, float scale) {
    constexpr int RP = Pitch<D>::row;
    constexpr int CH = kTile * D / 8 / kThreads;  // 16-byte chunks per thread per tile
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kTile * RP];  // K row-major
    __shared__ __attribute__((aligned(16))) uint16_t Vs[kTile * RP];  // V row-major

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + wave * 16 + c16;
    const bool qok = qrow < N;
    const int qcl = qok ? qrow : N - 1;
    const size_t ridx = (size_t)bh * N + qcl;

    bf16x8 qf[D / 32], uf[D / 32];
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
        qf[kc] = __builtin_bit_cast(bf16x8, ld_row16(Q + hoff, qrow, N, D, kc * 32 + 8 * g));
        uf[kc] = __builtin_bit_cast(bf16x8, ld_row16(dO + hoff, qrow, N, D, kc * 32 + 8 * g));
    }
    const float c = scale * kLog2e;
    const float lse2 = LSE[ridx] * kLog2e;
    const float Di = Drow[ridx];
    const bf16x8 ones = ones_row0(c16);

    f32x4 accA[D / 16], accB[GPROJ ? D / 16 : 1];
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) accA[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mb = 0; mb < (GPROJ ? D / 16 : 1); ++mb) accB[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 accR = {0.f, 0.f, 0.f, 0.f}, accM = {0.f, 0.f, 0.f, 0.f};

    const int nkv = causal ? min(T, tile + 1) : T;
    const bool q_tail = tile * kTile + kTile > N;

    u32x4 kreg[CH], vreg[CH];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            kreg[cI] = ld_row16(K + hoff, k0 + r, N, D, cc);
            vreg[cI] = ld_row16(V + hoff, k0 + r, N, D, cc);
        }
    };
    fetch(0);
    for (int kt = 0; kt < nkv; ++kt) {
        const int k0 = kt * kTile;
        __syncthreads();
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            *reinterpret_cast<u32x4*>(Ks + r * RP + cc) = kreg[cI];
            *reinterpret_cast<u32x4*>(Vs + r * RP + cc) = vreg[cI];
        }
        __syncthreads();
        if (kt + 1 < nkv) fetch(k0 + kTile);

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
        const bool edge = (causal && kt == tile) || q_tail || k0 + kTile > N;
        if (edge)
            dq_probs<true>(s, dp, c, lse2, Di, k0, g, qrow, qok, N, causal, tf, rf);
        else
            dq_probs<false>(s, dp, c, lse2, Di, k0, g, qrow, qok, N, causal, tf, rf);

        // A^T[d][query] += K^T[d][key] t^T[key][query]  (and B^T with r); the
        // row sums rho, m come from a constant ones operand.
#pragma unroll
        for (int kc2 = 0; kc2 < 2; ++kc2) {
#pragma unroll
            for (int mb = 0; mb < D / 16; ++mb) {
                const bf16x8 ka = ld_tr_operand(Ks, RP, kc2 * 32, mb * 16, c16, g);
                accA[mb] = mfma_16x16x32(ka, tf[kc2], accA[mb]);
                if (GPROJ) accB[mb] = mfma_16x16x32(ka, rf[kc2], accB[mb]);
            }
            if (GPROJ) {
                accR = mfma_16x16x32(ones, tf[kc2], accR);
                accM = mfma_16x16x32(ones, rf[kc2], accM);
            }
        }
    }

    // rho and m of this lane's query sit in accumulator row 0 (lanes g == 0).
    float lam = 0.f, rho = 0.f, msum = 0.f;
    if (GPROJ) {
        rho = __shfl(accR[0], c16);
        msum = __shfl(accM[0], c16);
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
            rho_out[ridx] = rho;
            m_out[ridx] = msum;
            lam_out[ridx] = lam;
        }
    }
}

// ----------------------------------------------------------- key-major pass
// P, r, t for one query tile of the key-major pass: lane holds queries 4g+i of
// each 16-query block for its key.
template <bool MASK>
__device__ __forceinline__ void dkdv_probs(const f32x4 (&s)[4], const f32x4 (&dp)[4],
                                           const f32x4 (&l2)[4], const f32x4 (&dd)[4], float c,
                                           int q0, int g, int krow, int N, int causal,
                                           bf16x8 (&tf)[2], bf16x8 (&rf)[2]) {
#pragma unroll
    for (int mq = 0; mq < 4; ++mq)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float P = fexp2(fmaf(s[mq][i], c, -l2[mq][i]));
            if constexpr (MASK) {
                const int query = q0 + mq * 16 + 4 * g + i;
                const bool ok = krow < N && query < N && (!causal || krow <= query);
                P = ok ? P : 0.f;
            }
            tf[mq >> 1][(mq & 1) * 4 + i] = to_bf16(P * (dp[mq][i] - dd[mq][i]));
            rf[mq >> 1][(mq & 1) * 4 + i] = to_bf16(P);
        }
}

template <int D, bool GPROJ>
__global__ __launch_bounds__(kThreads, D == 64 ? 2 : 1) void bwd_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow,
    const float* __restrict__ lam, uint16_t* __restrict__ dK, uint16_t* __restrict__ dV,
    int BH, int N, int causal, float scale) {
    constexpr int RP = Pitch<D>::row;
    constexpr int CH = kTile * D / 8 / kThreads;
    __shared__ __attribute__((aligned(16))) uint16_t Qs[kTile * RP];   // Q row-major
    __shared__ __attribute__((aligned(16))) uint16_t Us[kTile * RP];   // dO row-major
    __shared__ __attribute__((aligned(16))) uint16_t Zs[GPROJ ? kTile * RP : 8];  // BF16(lambda q)
    __shared__ __attribute__((aligned(16))) float lse2s[kTile];
    __shared__ __attribute__((aligned(16))) float Ds[kTile];

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, false, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const size_t soff = (size_t)bh * N;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int krow = tile * kTile + wave * 16 + c16;
    const bool kok = krow < N;

    // K^T and V^T as B operands: column = this lane's key, k = d.
    bf16x8 kf[D / 32], vf[D / 32];
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
        kf[kc] = __builtin_bit_cast(bf16x8, ld_row16(K + hoff, krow, N, D, kc * 32 + 8 * g));
        vf[kc] = __builtin_bit_cast(bf16x8, ld_row16(V + hoff, krow, N, D, kc * 32 + 8 * g));
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
    const bool k_tail = tile * kTile + kTile > N;

    u32x4 qreg[CH], ureg[CH];
    float lreg[CH];
    float lse_reg = 0.f, d_reg = 0.f;
    auto fetch = [&](int q0) {
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            qreg[cI] = ld_row16(Q + hoff, q0 + r, N, D, cc);
            ureg[cI] = ld_row16(dO + hoff, q0 + r, N, D, cc);
            if (GPROJ) lreg[cI] = lam[soff + min(q0 + r, N - 1)];
        }
        if (tid < kTile) {
            const int row = min(q0 + tid, N - 1);
            lse_reg = LSE[soff + row];
            d_reg = Drow[soff + row];
        }
    };
    fetch(qt0 * kTile);
    for (int qt = qt0; qt < T; ++qt) {
        const int q0 = qt * kTile;
        __syncthreads();
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
            const u32x4 qw = qreg[cI];
            *reinterpret_cast<u32x4*>(Qs + r * RP + cc) = qw;
            *reinterpret_cast<u32x4*>(Us + r * RP + cc) = ureg[cI];
            if (GPROJ) {
                // z = BF16(fl32(lambda q))
                u32x4 zw;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    zw[e] = (uint32_t)bf16_bits(lreg[cI] * lo_bf16(qw[e])) |
                            ((uint32_t)bf16_bits(lreg[cI] * hi_bf16(qw[e])) << 16);
                *reinterpret_cast<u32x4*>(Zs + r * RP + cc) = zw;
            }
        }
        if (tid < kTile) {
            lse2s[tid] = lse_reg * kLog2e;
            Ds[tid] = d_reg;
        }
        __syncthreads();
        if (qt + 1 < T) fetch(q0 + kTile);

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
        f32x4 l2[4], dd[4];
#pragma unroll
        for (int mq = 0; mq < 4; ++mq) {
            l2[mq] = *reinterpret_cast<const f32x4*>(lse2s + mq * 16 + 4 * g);
            dd[mq] = *reinterpret_cast<const f32x4*>(Ds + mq * 16 + 4 * g);
        }
        bf16x8 tf[2], rf[2];
        const bool edge = (causal && qt == tile) || k_tail || q0 + kTile > N;
        if (edge)
            dkdv_probs<true>(s, dp, l2, dd, c, q0, g, krow, N, causal, tf, rf);
        else
            dkdv_probs<false>(s, dp, l2, dd, c, q0, g, krow, N, causal, tf, rf);

        // dV^T[dv][key] += dO^T r ; dK^T += Q^T t ; C^T += Z^T r.
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb)
#pragma unroll
            for (int kc2 = 0; kc2 < 2; ++kc2) {
                accV[mb] = mfma_16x16x32(ld_tr_operand(Us, RP, kc2 * 32, mb * 16, c16, g), rf[kc2],
                                         accV[mb]);
                accK[mb] = mfma_16x16x32(ld_tr_operand(Qs, RP, kc2 * 32, mb * 16, c16, g), tf[kc2],
                                         accK[mb]);
                if (GPROJ)
                    accC[mb] = mfma_16x16x32(ld_tr_operand(Zs, RP, kc2 * 32, mb * 16, c16, g),
                                             rf[kc2], accC[mb]);
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
