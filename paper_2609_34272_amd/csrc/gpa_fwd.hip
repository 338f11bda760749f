// FA3-SBS attention forward on gfx950 bf16 MFMA (appendix "Implemented
// Arithmetic and Rounding", eq. gproj-forward): the exponent argument is
// fl32[ sub32(x, xmax) * fl32(alpha log2 e) ] with the unscaled logit x and the
// unscaled running row maximum xmax, so the largest logit maps to exactly
// exp2(0) = 1.
//
// Schedule: one workgroup per (batch*head, 64-query tile); 4 waves, each owning
// 16 queries.  K and V tiles of 64 keys are staged row-major in LDS (V is read
// back transposed with the LDS transpose load).  A wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16, so
// each lane holds 16 logits of ONE query (its column): the row maximum and the
// row sum are in-lane except for a 4-way exchange.  The probabilities are then
// already in the B-operand layout of O^T += V^T P^T, whose accumulator again
// keeps one query per lane, so the online-softmax rescale is a per-lane scalar.
#include "gpa_device.h"
#include "gpa_launch.h"

namespace gpa {
namespace {

template <int D>
__global__ __launch_bounds__(kThreads, GPA_FWD_OCC) void fwd_sbs_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O, float* __restrict__ LSE,
    int BH, int N, int causal, float scale) {
    constexpr int CH = kTile * D / 8 / kThreads;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[kTile * D];

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + wave * 16 + c16;
    const bool qok = qrow < N;

    // Q^T as the B operand: column = this lane's query, k = d.
    bf16x8 qf[D / 32];
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc)
        qf[kc] = __builtin_bit_cast(bf16x8, ld_row16(Q + hoff, qrow, N, D, kc * 32 + 8 * g));

    const float c = scale * kLog2e;  // fl32(alpha log2 e)
    float mrun = -INFINITY;          // running maximum of the unscaled logits
    float lrun = 0.f;                // this lane's share of the running sum of z
    f32x4 acc[D / 16];
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int kv_end = causal ? min(N, (tile + 1) * kTile) : N;
    const int nkv = (kv_end + kTile - 1) / kTile;

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
            *reinterpret_cast<u32x4*>(Ks + tile_off<D>(r, cc)) = kreg[cI];
            *reinterpret_cast<u32x4*>(Vs + tile_off<D>(r, cc)) = vreg[cI];
        }
        __syncthreads();
        if (kt + 1 < nkv) fetch(k0 + kTile);

        // S^T[key][query] for 4 blocks of 16 keys.
        f32x4 s[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < D / 32; ++kc)
                s[kb] = mfma_16x16x32(ld_b128(Ks + tile_off<D>(kb * 16 + c16, kc * 32 + 8 * g)), qf[kc],
                                      s[kb]);
        }
        // Only the diagonal tile and the key tail need masks (uniform branch).
        if ((causal && kt == tile) || k0 + kTile > N) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = k0 + kb * 16 + 4 * g + i;
                    const bool ok = key < N && (!causal || key <= qrow);
                    s[kb][i] = ok ? s[kb][i] : -INFINITY;
                }
        }
        float mx = s[0][0];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[kb][i]);
        mx = xor_max(mx);
        const float mnew = fmaxf(mrun, mx);
        // Rescale by exp2(fl32[fl32(mold - mnew) * c]): the same rule as z.
        // (mnew is finite: key 0 is visible to every row in tile 0.)
        const float corr = fexp2((mrun - mnew) * c);
        lrun *= corr;
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb) acc[mb] *= corr;

        bf16x8 pf[2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float z = fexp2((s[kb][i] - mnew) * c);
                lrun += z;
                pf[kb >> 1][(kb & 1) * 4 + i] = to_bf16(z);
            }
        mrun = mnew;

        // O^T[dv][query] += V^T[dv][key] P^T[key][query].
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb)
#pragma unroll
            for (int kc2 = 0; kc2 < 2; ++kc2)
                acc[mb] = mfma_16x16x32(ld_tr_operand<D>(Vs, kc2 * 32, mb * 16, c16, g), pf[kc2],
                                        acc[mb]);
    }

    const float ltot = xor_sum(lrun);
    if (qok) {
        uint16_t* orow = O + hoff + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < D / 16; ++mb)
            st_bf16x4(orow + mb * 16 + 4 * g, acc[mb][0] / ltot, acc[mb][1] / ltot,
                      acc[mb][2] / ltot, acc[mb][3] / ltot);
        if (g == 0) {
#pragma clang fp contract(off)
            const float lse = scale * mrun + logf(ltot);
            LSE[(size_t)bh * N + qrow] = lse;
        }
    }
}

}  // namespace

hipError_t launch_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, uint16_t* O,
                      float* LSE, const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    if (s.d == 64)
        fwd_sbs_kernel<64><<<grid, block, 0, st>>>(Q, K, V, O, LSE, s.BH, s.N, s.causal, s.scale);
    else
        fwd_sbs_kernel<128><<<grid, block, 0, st>>>(Q, K, V, O, LSE, s.BH, s.N, s.causal, s.scale);
    return hipGetLastError();
}

}  // namespace gpa
