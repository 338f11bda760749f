// FA3-SBS attention forward on gfx950 bf16 MFMA (appendix "Implemented
// Arithmetic and Rounding", eq. gproj-forward): the exponent argument is
// fl32[ sub32(x, xmax) * fl32(alpha log2 e) ] with the unscaled logit x and the
// unscaled running row maximum xmax, so the largest logit maps to exactly
// exp2(0) = 1.
//
// Schedule: one workgroup per (batch*head, 64-query tile); 4 waves.  Wave w
// owns 32 of the 64 queries (two 16-query MFMA blocks sharing every LDS
// fragment) and half of each 64-key tile; the two waves with the same queries
// merge their online-softmax states at the end with the same rescale rule.  K
// and V tiles are loaded straight into LDS (row-major, swizzled, double
// buffered); V is read back transposed with the LDS transpose load.  A wave
// computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16, so each lane holds the
// logits of ONE query (its column): the row maximum and sum are in-lane except
// for a 4-way exchange.  The probabilities are then already in the B-operand
// layout of O^T += V^T P^T, whose accumulator again keeps one query per lane,
// so the online-softmax rescale is a per-lane scalar.
#include "gpa_device.h"
#include "gpa_launch.h"

#include <type_traits>

namespace gpa {
namespace {

// Exponent argument of z = exp2(arg).  FA3-SBS (the path's forward):
// fl32[fl32(x - m) * c].  FMA (diagnostic only): the historical rounding
// fma(x, c, -fl32(m * c)), whose result is the rounding error of x*c rather
// than 0 when x = m (appendix on the source of the saved-output error, eq.
// historical-fma).
template <bool FMA>
__device__ __forceinline__ float exp_arg(float x, float m, float c) {
    if constexpr (FMA) {
#pragma clang fp contract(off)
        const float mc = m * c;
        return __builtin_fmaf(x, c, -mc);
    } else {
#pragma clang fp contract(off)
        return (x - m) * c;
    }
}

template <int D, bool FMA>
__global__ __launch_bounds__(kThreads, GPA_FWD_OCC) void fwd_sbs_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O, float* __restrict__ LSE,
    int BH, int Nmax, int causal, float scale, int G, const int* __restrict__ cu, int Hq,
    int total, const int* __restrict__ cu_k, int total_k, int Nkmax) {
    constexpr int MB = D / 16;
    constexpr int KC = D / 32;
    constexpr int PER_NB = MB * 4 + 2;  // acc, m, l of one query block
    // K and V tiles, double-buffered in two separate LDS objects so the
    // compiler can tell the tile being read from the one the DMA is filling.
    __shared__ __attribute__((aligned(16))) uint16_t KV0[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t KV1[2][kTile * D];

    const int T = (Nmax + kTile - 1) / kTile;  // tiles of the longest problem
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const SeqRows sr = seq_rows(cu, cu_k, bh, Nmax, Nkmax, G, Hq, total, total_k);
    const int N = sr.nq, Nk = sr.nk;
    if (tile * kTile >= N) return;  // a shorter sequence has no such tile
    const int off = Nk - N;           // causal: query i sees key j iff j <= i + off
    const size_t hoff = sr.q0 * D;    // query head: Q, O
    const size_t kvoff = sr.kv0 * D;  // its key/value head
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int qh = wave & 1;   // which 32 of the workgroup's 64 queries
    const int kh = wave >> 1;  // which 32 of each 64-key tile
    const int q0w = tile * kTile + 32 * qh;

    // Q^T as the B operand: column = this lane's query of block nb, k = d.
    const rsrc_t rq = make_rsrc(Q + hoff, (uint32_t)N * (2 * D));
    bf16x8 qf[2][KC];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
            qf[nb][kc] = __builtin_bit_cast(bf16x8, ld_row16<D>(rq, q0w + nb * 16 + c16, kc * 32 + 8 * g));

    const float c = scale * kLog2e;  // fl32(alpha log2 e)
    float mrun[2] = {-INFINITY, -INFINITY};  // running maximum of the unscaled logits
    float lrun[2] = {0.f, 0.f};              // this lane's share of the running sum of z
    f32x4 acc[2][MB];                        // O^T[dv][query]
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Only the last one or two key tiles need masks (the causal diagonal, the
    // key tail).
    const KeyRange kr = key_range(tile, Nk, off, causal);
    const int nkv = kr.nkv, nplain = kr.nplain;

    // Zero both buffers once, so that every value a product can read is finite
    // whatever the DMA leaves in the slots of rows beyond Nk (it writes zeros
    // there, but the tail does not depend on it).
    {
        u32x4* z0 = reinterpret_cast<u32x4*>(&KV0[0][0]);
        u32x4* z1 = reinterpret_cast<u32x4*>(&KV1[0][0]);
        constexpr int n16 = (int)(sizeof(KV0) / 16);
#pragma unroll
        for (int i = tid; i < n16; i += kThreads) {
            z0[i] = u32x4{0u, 0u, 0u, 0u};
            z1[i] = u32x4{0u, 0u, 0u, 0u};
        }
    }
    __syncthreads();

    TileDma<D> dma;
    dma.init(lane, wave);
    dma.load(K + kvoff, KV0[0], 0, Nk);
    dma.load(V + kvoff, KV0[1], 0, Nk);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    auto step = [&](auto masked, int kt, const uint16_t* Kc, const uint16_t* Vc, uint16_t* Kn,
                    uint16_t* Vn) {
        constexpr bool MASK = decltype(masked)::value;
        const int k0 = kt * kTile;
        if (kt + 1 < nkv) {
            dma.load(K + kvoff, Kn, k0 + kTile, Nk);
            dma.load(V + kvoff, Vn, k0 + kTile, Nk);
        }
        // Keep the loads of the next tile at the top of the step: left alone,
        // the scheduler sinks them next to the closing wait, which exposes
        // their whole latency.
        __builtin_amdgcn_sched_barrier(0);
        // S^T[key][query] for this wave's 32 keys x 32 queries; s[nb][kb]
        // holds keys 4g+i of key block kb for query block nb.  The wave raises
        // its issue priority while it feeds the matrix core, so that the other
        // wave on the SIMD runs its exponentials meanwhile (h16_n4096_d128
        // forward 6 % faster; neutral on the batched d = 128 workload).
        __builtin_amdgcn_s_setprio(1);
        f32x4 s[2][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[0][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
            s[1][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const bf16x8 ka = ld_b128(Kc + tile_off<D>(32 * kh + kb * 16 + c16, kc * 32 + 8 * g));
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) s[nb][kb] = mfma_16x16x32(ka, qf[nb][kc], s[nb][kb]);
            }
        }
        if constexpr (MASK) {
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = k0 + 32 * kh + kb * 16 + 4 * g + i;
                        const int qrow = q0w + nb * 16 + c16;
                        const bool ok = key < Nk && (!causal || key <= qrow + off);
                        s[nb][kb][i] = ok ? s[nb][kb][i] : -INFINITY;
                    }
        }
        __builtin_amdgcn_s_setprio(0);
        bf16x8 pf[2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            float mx = s[nb][0][0];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[nb][kb][i]);
            mx = xor_max(mx);
            const float mnew = fmaxf(mrun[nb], mx);
            // A wave half may not have seen a visible key yet (mnew = -inf);
            // then every z is 0 and nothing is rescaled.
            const float ms = (mnew == -INFINITY) ? 0.f : mnew;
            // Rescale by exp2(fl32[fl32(mold - mnew) * c]): the same rule as z;
            // skipped when no query of the wave has a new maximum (corr is then
            // exactly 1).
            if (__builtin_amdgcn_ballot_w64(mnew != mrun[nb]) != 0) {
                const float corr = fexp2((mrun[nb] - ms) * c);
                lrun[nb] *= corr;
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) acc[nb][mb] *= corr;
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float z = fexp2(exp_arg<FMA>(s[nb][kb][i], ms, c));
                    lrun[nb] += z;
                    pf[nb][kb * 4 + i] = to_bf16(z);
                }
            mrun[nb] = mnew;
        }
        // O^T[dv][query] += V^T[dv][key] P^T[key][query].
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const bf16x8 va = ld_tr_operand<D>(Vc, 32 * kh, mb * 16, c16, g);
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) acc[nb][mb] = mfma_16x16x32(va, pf[nb], acc[nb][mb]);
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the next tile
        __syncthreads();
    };
    const std::false_type plain;
    const std::true_type masked;
    int kt = 0;
    for (; kt + 1 < nplain; kt += 2) {
        step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
        step(plain, kt + 1, KV1[0], KV1[1], KV0[0], KV0[1]);
    }
    if (kt < nplain) {
        step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
        ++kt;
    }
    // Tile kt lives in buffer kt mod 2.
    for (; kt < nkv; ++kt) {
        if (kt & 1)
            step(masked, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else
            step(masked, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }

    // Merge the two key halves of each query (waves w and w + 2): waves 2, 3
    // park (acc, m, l) in LDS, waves 0, 1 combine them with the same rescale
    // rule and finish.
    // Query block nb goes through buffer object nb (each holds 2 x 64 x PER_NB
    // floats).
    static_assert(sizeof(KV0) >= 2 * 64 * PER_NB * sizeof(float), "merge space");
    float* const scratch[2] = {reinterpret_cast<float*>(&KV0[0][0]),
                               reinterpret_cast<float*>(&KV1[0][0])};
    if (wave >= 2) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            float* p = scratch[nb] + (wave - 2) * 64 * PER_NB + lane;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) p[(mb * 4 + i) * 64] = acc[nb][mb][i];
            p[(MB * 4) * 64] = mrun[nb];
            p[(MB * 4 + 1) * 64] = lrun[nb];
        }
    }
    __syncthreads();
    if (wave >= 2) return;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const float* p = scratch[nb] + wave * 64 * PER_NB + lane;
        const float mo = p[(MB * 4) * 64];
        const float lo = p[(MB * 4 + 1) * 64];
        const float mt = fmaxf(mrun[nb], mo);
        const float ms = (mt == -INFINITY) ? 0.f : mt;
        const float fa = fexp2((mrun[nb] - ms) * c);
        const float fb = fexp2((mo - ms) * c);
        const float ltot = xor_sum(lrun[nb] * fa + lo * fb);
        const int qrow = q0w + nb * 16 + c16;
        if (qrow < N) {
            // A query that sees no key (l = 0; a visible key adds z = 1) gets
            // O = 0 and LSE = +inf, so the backward's P is 0 on its row.  l is
            // +0 exactly then; the test is on the bits so that a NaN row (NaN
            // l) keeps NaN outputs whatever the compiler assumes about NaNs.
            const bool empty = __float_as_uint(ltot) == 0u;
            uint16_t* orow = O + hoff + (size_t)qrow * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    v[i] = empty ? 0.f : (acc[nb][mb][i] * fa + p[(mb * 4 + i) * 64] * fb) / ltot;
                st_bf16x4(orow + mb * 16 + 4 * g, v[0], v[1], v[2], v[3]);
            }
            if (g == 0) {
#pragma clang fp contract(off)
                const float lse = scale * mt + logf(ltot);
                LSE[sr.q0 + qrow] = empty ? INFINITY : lse;
            }
        }
    }
}

// Variant with one 16-query block per wave: each of the 4 waves owns 16 of
// the workgroup's 64 queries and runs them against the whole 64-key tile, so
// the online-softmax bookkeeping (row maximum, rescale of the output
// accumulator, correction factor) is paid once per 64 keys and no merge of
// partial states is needed; the price is that every K and V fragment read from
// LDS feeds one MFMA instead of two.  Fewer registers per wave allow more
// waves per SIMD.  The arithmetic per (query, key) is that of fwd_sbs_kernel.
template <int D, bool FMA>
__global__ __launch_bounds__(kThreads, GPA_FWD16_OCC) void fwd_sbs_q16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O, float* __restrict__ LSE,
    int BH, int Nmax, int causal, float scale, int G, const int* __restrict__ cu, int Hq,
    int total, const int* __restrict__ cu_k, int total_k, int Nkmax) {
    constexpr int MB = D / 16;
    constexpr int KC = D / 32;
    __shared__ __attribute__((aligned(16))) uint16_t KV0[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t KV1[2][kTile * D];

    const int T = (Nmax + kTile - 1) / kTile;  // tiles of the longest problem
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile, GPA_FWD16_OCC);
    const SeqRows sr = seq_rows(cu, cu_k, bh, Nmax, Nkmax, G, Hq, total, total_k);
    const int N = sr.nq, Nk = sr.nk;
    if (tile * kTile >= N) return;  // a shorter sequence has no such tile
    const int off = Nk - N;  // causal: query i sees key j iff j <= i + off
    const size_t hoff = sr.q0 * D;
    const size_t kvoff = sr.kv0 * D;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + 16 * wave + c16;  // this lane's query

    const rsrc_t rq = make_rsrc(Q + hoff, (uint32_t)N * (2 * D));
    bf16x8 qf[KC];
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
        qf[kc] = __builtin_bit_cast(bf16x8, ld_row16<D>(rq, qrow, kc * 32 + 8 * g));

    const float c = scale * kLog2e;
    float mrun = -INFINITY, lrun = 0.f;
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const KeyRange kr = key_range(tile, Nk, off, causal);
    const int nkv = kr.nkv, nplain = kr.nplain;

    TileDma<D> dma;
    dma.init(lane, wave);
    wait_vm_lgkm0<0>();
    dma.load(K + kvoff, KV0[0], 0, Nk);
    dma.load(V + kvoff, KV0[1], 0, Nk);
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();

    auto step = [&](auto masked, int kt, const uint16_t* Kc, const uint16_t* Vc, uint16_t* Kn,
                    uint16_t* Vn) {
        constexpr bool MASK = decltype(masked)::value;
        const int k0 = kt * kTile;
        if (kt + 1 < nkv) {
            dma.load(K + kvoff, Kn, k0 + kTile, Nk);
            dma.load(V + kvoff, Vn, k0 + kTile, Nk);
        }
        __builtin_amdgcn_sched_barrier(0);
        // S^T[key][query]: s[kb] holds keys 16 kb + 4g + i for this lane's query.
        f32x4 s[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < KC; ++kc)
                s[kb] = mfma_16x16x32(ld_b128(Kc + tile_off<D>(kb * 16 + c16, kc * 32 + 8 * g)),
                                      qf[kc], s[kb]);
        }
        if constexpr (MASK) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = k0 + kb * 16 + 4 * g + i;
                    const bool ok = key < Nk && (!causal || key <= qrow + off);
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
        const float ms = (mnew == -INFINITY) ? 0.f : mnew;
        // Rescale only when some query of the wave has a new maximum: otherwise
        // corr is exactly 1 in every lane and multiplying by it changes nothing.
        if (__builtin_amdgcn_ballot_w64(mnew != mrun) != 0) {
            const float corr = fexp2((mrun - ms) * c);
            lrun *= corr;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[mb] *= corr;
        }
        // pf[j]: B operand of keys 32 j .. 32 j + 31 (k-layout {4g+i, 16+4g+i}).
        bf16x8 pf[2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float z = fexp2(exp_arg<FMA>(s[kb][i], ms, c));
                lrun += z;
                pf[kb >> 1][(kb & 1) * 4 + i] = to_bf16(z);
            }
        mrun = mnew;
        // O^T[dv][query] += V^T[dv][key] P^T[key][query].
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[mb] = mfma_16x16x32(ld_tr_operand<D>(Vc, 32 * j, mb * 16, c16, g), pf[j],
                                        acc[mb]);
        wait_vm_lgkm0<0>();
        __builtin_amdgcn_s_barrier();
    };
    const std::false_type plain;
    const std::true_type masked;
    int kt = 0;
    for (; kt + 1 < nplain; kt += 2) {
        step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
        step(plain, kt + 1, KV1[0], KV1[1], KV0[0], KV0[1]);
    }
    if (kt < nplain) {
        step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
        ++kt;
    }
    // Tile kt lives in buffer kt mod 2.
    for (; kt < nkv; ++kt) {
        if (kt & 1)
            step(masked, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else
            step(masked, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }

    const float ltot = xor_sum(lrun);
    if (qrow < N) {
        // A query that sees no key (l = 0; a visible key adds z = 1) gets O = 0
        // and LSE = +inf, so the backward's P is 0 on its row.  l is +0 exactly
        // then; the test is on the bits so that a NaN row (NaN l) keeps NaN
        // outputs whatever the compiler assumes about NaNs.
        const bool empty = __float_as_uint(ltot) == 0u;
        uint16_t* orow = O + hoff + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = empty ? 0.f : acc[mb][i] / ltot;
            st_bf16x4(orow + mb * 16 + 4 * g, v[0], v[1], v[2], v[3]);
        }
        if (g == 0) {
#pragma clang fp contract(off)
            const float lse = scale * mrun + logf(ltot);
            LSE[sr.q0 + qrow] = empty ? INFINITY : lse;
        }
    }
}

}  // namespace

hipError_t launch_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, uint16_t* O,
                      float* LSE, const Shape& s, hipStream_t st, bool fma_forward) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    // d = 64: one 16-query block per wave (measured faster); d = 128: two
    // blocks per wave, whose halved LDS reads matter more there.
#define GPA_FWD(KERNEL, DD, FM)                                                               \
    launch_kernel(KERNEL<DD, FM>, grid, block, st, Q, K, V, O, LSE, s.BH, s.N, s.causal,      \
                  s.scale, s.G, s.cu, s.Hq, s.total, s.cu_k, s.total_k, s.Nk > 0 ? s.Nk : s.N)
    if (s.d == 64) {
        if (fma_forward) GPA_FWD(fwd_sbs_q16_kernel, 64, true);
        else GPA_FWD(fwd_sbs_q16_kernel, 64, false);
    } else {
        if (fma_forward) GPA_FWD(fwd_sbs_kernel, 128, true);
        else GPA_FWD(fwd_sbs_kernel, 128, false);
    }
#undef GPA_FWD
    return hipGetLastError();
}

}  // namespace gpa
