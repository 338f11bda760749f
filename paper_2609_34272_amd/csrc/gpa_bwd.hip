// Attention backward with the GProj correction on gfx950 bf16 MFMA
// (Algorithm 1; appendix "Implemented Arithmetic and Rounding", eqs.
// gproj-row-mass, gproj-accumulators, gproj-query-implemented,
// gproj-key-implemented).
//
// Schedule (deterministic, no atomics).  Algorithm 1 accumulates dQ and B = rK
// with atomic adds from a key-major loop and then needs a second key-major pass
// for dK, because lambda_i = rho_i / m_i is known only after row i has seen
// every key.  Here the same arithmetic is split by ownership instead:
//   1. bwd_dq    : query-major.  A workgroup owns 64 query rows and streams the
//                  key tiles, so A = tK, B = rK, rho and m stay in registers; at
//                  the end it forms lambda = rho/m once and writes
//                  dQ = BF16(fl32[alpha (A - lambda B)]) and lambda.
//                  In gproj mode it also writes z = BF16(lambda q), once per row.
//                  It also forms D_i = rowsum(dO_i * O_i) (FP32) for its rows.
//   2. bwd_dkdv  : key-major.  A workgroup owns 64 keys and streams the query
//                  tiles (Q, dO and z); with lambda already applied it
//                  accumulates dV = r^T dO, dK^acc = t^T Q and C = r^T z and
//                  writes dK = BF16(fl32[alpha (dK^acc - C)]).
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


// --------------------------------------------------------- query-major pass
// P, r, t for 32 keys (two 16-key blocks) of the query-major pass: lane holds
// keys 4g+i of each block for its query.  MASK applies the causal and tail
// masks (only diagonal and tail tiles need them).
template <bool MASK>
__device__ __forceinline__ void dq_probs(const f32x4 (&s)[2], const f32x4 (&dp)[2], float c,
                                         float lse2, float Di, int key0, int g, int qrow,
                                         bool qok, int N, int causal, bf16x8& tf, bf16x8& rf) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float P = fexp2(fmaf(s[kb][i], c, -lse2));
            if constexpr (MASK) {
                const int key = key0 + kb * 16 + 4 * g + i;
                const bool ok = qok && key < N && (!causal || key <= qrow);
                P = ok ? P : 0.f;
            }
            tf[kb * 4 + i] = to_bf16(P * (dp[kb][i] - Di));
            rf[kb * 4 + i] = to_bf16(P);
        }
}

// Stage one 64-row tile of up to three BF16 tensors (global -> registers ->
// swizzled LDS).  Rows at or beyond N are zero.
template <int D, int NT>
struct TileStager {
    static constexpr int CH = kTile * D / 8 / kThreads;  // 16-byte chunks per thread
    u32x4 reg[NT][CH];

    __device__ __forceinline__ void fetch(const uint16_t* const (&src)[NT], int row0, int N,
                                          int tid) {
        const bool full = row0 + kTile <= N;
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
#pragma unroll
            for (int t = 0; t < NT; ++t)
                reg[t][cI] = full ? *reinterpret_cast<const u32x4*>(src[t] + (size_t)(row0 + r) * D + cc)
                                  : ld_row16(src[t], row0 + r, N, D, cc);
        }
    }
    __device__ __forceinline__ void store(uint16_t* const (&dst)[NT], int tid) const {
#pragma unroll
        for (int cI = 0; cI < CH; ++cI) {
            const int ch = tid + cI * kThreads;
            const int r = ch / (D / 8);
            const int cc = (ch - r * (D / 8)) * 8;
#pragma unroll
            for (int t = 0; t < NT; ++t)
                *reinterpret_cast<u32x4*>(dst[t] + tile_off<D>(r, cc)) = reg[t][cI];
        }
    }
};

template <int D, bool GPROJ, bool WRITE_Z>
__global__ __launch_bounds__(kThreads, D == 64 ? GPA_DQ_OCC64 : 2) void bwd_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ O,
    const uint16_t* __restrict__ dO, const float* __restrict__ LSE, float* __restrict__ D_out,
    uint16_t* __restrict__ dQ, float* __restrict__ rho_out, float* __restrict__ m_out,
    float* __restrict__ lam_out, uint16_t* __restrict__ Zout, int BH, int N, int causal,
    float scale) {
    // Double-buffered K and V tiles (row-major, swizzled).
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[2][kTile * D];

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
    // Algorithm 1's preprocessing, fused: D_i = sum_c fl32(dO_ic O_ic) (BF16 x BF16
    // products are exact in FP32), from this lane's column slices of the row,
    // summed over the row's 4 lanes.  The key-major pass reads D back.
    float dpart = 0.f;
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
        const u32x4 ow = ld_row16(O + hoff, qrow, N, D, kc * 32 + 8 * g);
        const u32x4 uw = __builtin_bit_cast(u32x4, uf[kc]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            dpart += lo_bf16(uw[e]) * lo_bf16(ow[e]);
            dpart += hi_bf16(uw[e]) * hi_bf16(ow[e]);
        }
    }
    const float Di = xor_sum(dpart);
    const float c = scale * kLog2e;
    const float lse2 = LSE[ridx] * kLog2e;
    const bf16x8 ones = ones_row0(c16);

    f32x4 accA[D / 16], accB[GPROJ ? D / 16 : 1];
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) accA[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mb = 0; mb < (GPROJ ? D / 16 : 1); ++mb) accB[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 accR = {0.f, 0.f, 0.f, 0.f}, accM = {0.f, 0.f, 0.f, 0.f};

    const int nkv = causal ? min(T, tile + 1) : T;
    const bool q_tail = tile * kTile + kTile > N;

    TileStager<D, 2> st;
    const uint16_t* const src[2] = {K + hoff, V + hoff};
    st.fetch(src, 0, N, tid);
    {
        uint16_t* const dst[2] = {Ks[0], Vs[0]};
        st.store(dst, tid);
    }
    __syncthreads();
    for (int kt = 0; kt < nkv; ++kt) {
        const int k0 = kt * kTile;
        const int cur = kt & 1;
        if (kt + 1 < nkv) st.fetch(src, k0 + kTile, N, tid);
        const uint16_t* Kc = Ks[cur];
        const uint16_t* Vc = Vs[cur];
        const bool edge = (causal && kt == tile) || q_tail || k0 + kTile > N;

        // Two halves of 32 keys.  S^T = K Q^T and dP^T = V dO^T leave each lane
        // with keys 4g+i of each 16-key block for its own query.
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4 s[2], dp[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int kb = 2 * h + b;
                s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
                dp[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kc = 0; kc < D / 32; ++kc) {
                    s[b] = mfma_16x16x32(ld_b128(Kc + tile_off<D>(kb * 16 + c16, kc * 32 + 8 * g)),
                                         qf[kc], s[b]);
                    dp[b] = mfma_16x16x32(ld_b128(Vc + tile_off<D>(kb * 16 + c16, kc * 32 + 8 * g)),
                                          uf[kc], dp[b]);
                }
            }
            bf16x8 tf, rf;
            if (edge)
                dq_probs<true>(s, dp, c, lse2, Di, k0 + 32 * h, g, qrow, qok, N, causal, tf, rf);
            else
                dq_probs<false>(s, dp, c, lse2, Di, k0 + 32 * h, g, qrow, qok, N, causal, tf, rf);
            // A^T[d][query] += K^T[d][key] t^T[key][query] (and B^T with r); the
            // row sums rho, m come from a constant ones operand.
#pragma unroll
            for (int mb = 0; mb < D / 16; ++mb) {
                const bf16x8 ka = ld_tr_operand<D>(Kc, h * 32, mb * 16, c16, g);
                accA[mb] = mfma_16x16x32(ka, tf, accA[mb]);
                if (GPROJ) accB[mb] = mfma_16x16x32(ka, rf, accB[mb]);
            }
            if (GPROJ) {
                accR = mfma_16x16x32(ones, tf, accR);
                accM = mfma_16x16x32(ones, rf, accM);
            }
        }
        if (kt + 1 < nkv) {
            uint16_t* const dst[2] = {Ks[cur ^ 1], Vs[cur ^ 1]};
            st.store(dst, tid);
        }
        __syncthreads();
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
        if (WRITE_Z) {
            // z = BF16(fl32(lambda q)) for the key correction: the lane holds
            // d = kc*32 + 8g .. +7 of its query row.
#pragma unroll
            for (int kc = 0; kc < D / 32; ++kc) {
                bf16x8 z;
#pragma unroll
                for (int e = 0; e < 8; ++e) z[e] = to_bf16(lam * bf16_to_f32(qf[kc][e]));
                *reinterpret_cast<bf16x8*>(Zout + hoff + (size_t)qrow * D + kc * 32 + 8 * g) = z;
            }
        }
        if (g == 0) {
            D_out[ridx] = Di;
            rho_out[ridx] = rho;
            m_out[ridx] = msum;
            lam_out[ridx] = lam;
        }
    }
}

// ----------------------------------------------------------- key-major pass
// P, r, t for 32 queries (two 16-query blocks) of the key-major pass: lane
// holds queries 4g+i of each block for its key.
template <bool MASK>
__device__ __forceinline__ void dkdv_probs(const f32x4 (&s)[2], const f32x4 (&dp)[2],
                                           const f32x4 (&l2)[2], const f32x4 (&dd)[2], float c,
                                           int qb0, int g, int krow, int N, int causal,
                                           bf16x8& tf, bf16x8& rf) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float P = fexp2(fmaf(s[b][i], c, -l2[b][i]));
            if constexpr (MASK) {
                const int query = qb0 + b * 16 + 4 * g + i;
                const bool ok = krow < N && query < N && (!causal || krow <= query);
                P = ok ? P : 0.f;
            }
            tf[b * 4 + i] = to_bf16(P * (dp[b][i] - dd[b][i]));
            rf[b * 4 + i] = to_bf16(P);
        }
}

template <int D, bool GPROJ>
__global__ __launch_bounds__(kThreads, D == 64 ? GPA_DKDV_OCC64 : 1) void bwd_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow,
    const uint16_t* __restrict__ Z, uint16_t* __restrict__ dK, uint16_t* __restrict__ dV,
    int BH, int N, int causal, float scale) {
    constexpr int NT = GPROJ ? 3 : 2;  // staged tensors: Q, dO (and Z = BF16(lambda Q))
    __shared__ __attribute__((aligned(16))) uint16_t Ts[2][NT][kTile * D];
    __shared__ __attribute__((aligned(16))) float lse2s[2][kTile];
    __shared__ __attribute__((aligned(16))) float Ds[2][kTile];

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

    TileStager<D, NT> st;
    const uint16_t* src[NT];
    src[0] = Q + hoff;
    src[1] = dO + hoff;
    if (GPROJ) src[NT - 1] = Z + hoff;
    float lse_reg = 0.f, d_reg = 0.f;
    auto fetch_stats = [&](int q0) {
        if (tid < kTile) {
            const int row = min(q0 + tid, N - 1);
            lse_reg = LSE[soff + row];
            d_reg = Drow[soff + row];
        }
    };
    auto store = [&](int buf) {
        uint16_t* dst[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) dst[t] = Ts[buf][t];
        st.store(dst, tid);
        if (tid < kTile) {
            lse2s[buf][tid] = lse_reg * kLog2e;
            Ds[buf][tid] = d_reg;
        }
    };
    st.fetch(src, qt0 * kTile, N, tid);
    fetch_stats(qt0 * kTile);
    store(0);
    __syncthreads();
    for (int qt = qt0; qt < T; ++qt) {
        const int q0 = qt * kTile;
        const int cur = (qt - qt0) & 1;
        if (qt + 1 < T) {
            st.fetch(src, q0 + kTile, N, tid);
            fetch_stats(q0 + kTile);
        }
        const uint16_t* Qc = Ts[cur][0];
        const uint16_t* Uc = Ts[cur][1];
        const uint16_t* Zc = Ts[cur][NT - 1];
        const bool edge = (causal && qt == tile) || k_tail || q0 + kTile > N;

        // Two halves of 32 queries.  S = Q K^T and dP = dO V^T leave each lane
        // with queries 4g+i of each 16-query block for its own key.
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4 s[2], dp[2], l2[2], dd[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int mq = 2 * h + b;
                s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
                dp[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kc = 0; kc < D / 32; ++kc) {
                    s[b] = mfma_16x16x32(ld_b128(Qc + tile_off<D>(mq * 16 + c16, kc * 32 + 8 * g)),
                                         kf[kc], s[b]);
                    dp[b] = mfma_16x16x32(ld_b128(Uc + tile_off<D>(mq * 16 + c16, kc * 32 + 8 * g)),
                                          vf[kc], dp[b]);
                }
                l2[b] = *reinterpret_cast<const f32x4*>(&lse2s[cur][mq * 16 + 4 * g]);
                dd[b] = *reinterpret_cast<const f32x4*>(&Ds[cur][mq * 16 + 4 * g]);
            }
            bf16x8 tf, rf;
            if (edge)
                dkdv_probs<true>(s, dp, l2, dd, c, q0 + 32 * h, g, krow, N, causal, tf, rf);
            else
                dkdv_probs<false>(s, dp, l2, dd, c, q0 + 32 * h, g, krow, N, causal, tf, rf);
            // dV^T[dv][key] += dO^T r ; dK^T += Q^T t ; C^T += Z^T r.
#pragma unroll
            for (int mb = 0; mb < D / 16; ++mb) {
                accV[mb] = mfma_16x16x32(ld_tr_operand<D>(Uc, h * 32, mb * 16, c16, g), rf, accV[mb]);
                accK[mb] = mfma_16x16x32(ld_tr_operand<D>(Qc, h * 32, mb * 16, c16, g), tf, accK[mb]);
                if (GPROJ)
                    accC[mb] = mfma_16x16x32(ld_tr_operand<D>(Zc, h * 32, mb * 16, c16, g), rf,
                                             accC[mb]);
            }
        }
        if (qt + 1 < T) store(cur ^ 1);
        __syncthreads();
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

hipError_t launch_bwd_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* O, const uint16_t* dO, const float* LSE, float* Drow,
                         uint16_t* dQ, float* rho, float* msum, float* lambda, uint16_t* Z,
                         int mode, const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
#define GPA_DQ(DD, GP, WZ)                                                                  \
    bwd_dq_kernel<DD, GP, WZ><<<grid, block, 0, st>>>(Q, K, V, O, dO, LSE, Drow, dQ, rho, msum, \
                                                      lambda, Z, s.BH, s.N, s.causal, s.scale)
    if (s.d == 64) {
        if (mode == 2) GPA_DQ(64, true, true);
        else if (mode == 1) GPA_DQ(64, true, false);
        else GPA_DQ(64, false, false);
    } else {
        if (mode == 2) GPA_DQ(128, true, true);
        else if (mode == 1) GPA_DQ(128, true, false);
        else GPA_DQ(128, false, false);
    }
#undef GPA_DQ
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* LSE, const float* Drow,
                           const uint16_t* Z, uint16_t* dK, uint16_t* dV, int mode,
                           const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    const bool gp = mode == 2;
#define GPA_DKDV(DD, GP)                                                             \
    bwd_dkdv_kernel<DD, GP><<<grid, block, 0, st>>>(Q, K, V, dO, LSE, Drow, Z, dK, dV, \
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
