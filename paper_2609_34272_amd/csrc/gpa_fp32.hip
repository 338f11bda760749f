// Fused FP32 attention baseline on gfx950: BF16 inputs and outputs, every
// product and accumulation in FP32 (appendix "Comparison Methods", "Fused
// FP32 baseline").  The forward saves FP32 O and three FP32 row statistics --
// the LSE, the row maximum and the inverse normaliser -- and the backward
// rebuilds P = exp(s - rowmax) * (1/l) from the last two, which keeps the
// normalisation exact to FP32 where large logits leave the LSE short of
// resolution.  No N x N matrix is stored.
//
// The paper's kernel is SIMT FP32 because the Hopper tensor cores round FP32
// operands to TF32.  gfx950's matrix cores have a true FP32 mode
// (v_mfma_f32_16x16x4_f32: FP32 operands, FP32 products and accumulation, no
// reduced-precision step), so the contractions run there; the softmax, its
// statistics and the score gradient run on the vector ALU in FP32.  The
// inputs are BF16, so decoding them to FP32 is exact.
//
// MFMA layout (16x16x4, FP32, wave64): lane (c16 = lane & 15, g = lane >> 4)
// supplies A[c16][g] and B[g][c16]; the accumulator holds D[4g + i][c16].  A
// 16 x 16 product over k = d is the sum of d/4 such MFMAs; step s of it lets
// lane g contract d index dk(s) = 64 (s / 16) + 16 g + s % 16, a permutation
// shared by both operands, so each lane reads 16 consecutive values of its
// row (two 16-byte LDS reads) per 64 columns.  The accumulator of S^T = K Q^T
// (or S = Q K^T) leaves each lane the values of rows 4g + i of its column;
// fed back one element i at a time as the B operand of the next product, they
// pair with A elements of rows 4g + i, which the gfx950 LDS transpose read
// delivers from a row-major BF16 tile.  P and dS never pass through LDS.
//
// Work split: a workgroup has 4 waves and owns 64 rows (queries in the
// forward and the query-major pass, keys in the key-major pass), 16 per wave;
// it streams 64-row tiles of the other side through a double-buffered LDS
// ring filled with the LDS DMA load.
#include "gpa_device.h"
#include "gpa_launch.h"

#include <type_traits>

namespace gpa {
namespace {

__device__ __forceinline__ f32x4 mfma_f32(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Per query tile, the key-major pass reads three 64-float blocks: the scaled
// row maximum (+inf beyond N, so P = 0 there), the inverse normaliser (0
// beyond N) and D = rowsum(dO O32) (0 beyond N).
constexpr int kF32Stat = 3 * kTile;

// 16 consecutive BF16 values of row `row` at column `col` of a swizzled LDS
// tile, widened exactly to FP32.
template <int D>
__device__ __forceinline__ void lds_row16(const uint16_t* X, int row, int col, float (&out)[16]) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(X + tile_off<D>(row, col));
    const u32x4 b = *reinterpret_cast<const u32x4*>(X + tile_off<D>(row, col + 8));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        out[2 * e] = lo_bf16(a[e]);
        out[2 * e + 1] = hi_bf16(a[e]);
        out[8 + 2 * e] = lo_bf16(b[e]);
        out[8 + 2 * e + 1] = hi_bf16(b[e]);
    }
}

// A row of a [N, D] BF16 tensor in the permuted k order: out[s] = X[row][dk(s)]
// (zero beyond N through the buffer resource).
template <int D>
__device__ __forceinline__ void ld_row_perm(rsrc_t r, int row, int g, float (&out)[D / 4]) {
#pragma unroll
    for (int h = 0; h < D / 64; ++h) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const u32x4 w = ld_row16<D>(r, row, 64 * h + 16 * g + 8 * p);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                out[16 * h + 8 * p + 2 * e] = lo_bf16(w[e]);
                out[16 * h + 8 * p + 2 * e + 1] = hi_bf16(w[e]);
            }
        }
    }
}

// One 16 x 16 block X_rows . Y^T over d: the A side comes from a swizzled LDS
// tile (rows r0 + c16), the B side from registers in the permuted order.
template <int D>
__device__ __forceinline__ f32x4 block_dot(const uint16_t* X, int r0, const float (&y)[D / 4],
                                           int c16, int g) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < D / 64; ++h) {
        float a[16];
        lds_row16<D>(X, r0 + c16, 64 * h + 16 * g, a);
#pragma unroll
        for (int s = 0; s < 16; ++s) acc = mfma_f32(a[s], y[16 * h + s], acc);
    }
    return acc;
}

// acc[mb] += X^T[d][rows] . B[rows][col] for the 64 tile rows, where the B
// values b[kb][i] belong to row 16 kb + 4 g + i and X is a row-major
// swizzled BF16 tile: the transpose read gives lane (c16, g) X[32 kb2 + 4 g +
// r][16 mb + c16] and X[32 kb2 + 16 + 4 g + r][...] for r = 0..3.
template <int D>
__device__ __forceinline__ void tr_accumulate(const uint16_t* X, const f32x4 (&b)[4],
                                              f32x4 (&acc)[D / 16], int c16, int g) {
#pragma unroll
    for (int mb = 0; mb < D / 16; ++mb) {
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2) {
            const bf16x8 t = ld_tr_operand<D>(X, 32 * kb2, 16 * mb, c16, g);
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[mb] = mfma_f32(bf16_to_f32(t[4 * half + i]), b[2 * kb2 + half][i], acc[mb]);
        }
    }
}

// ------------------------------------------------------------------ forward
template <int D>
__global__ __launch_bounds__(kThreads, 2) void f32_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ O32, uint16_t* __restrict__ O,
    float* __restrict__ LSE, float* __restrict__ Mrow, float* __restrict__ Linv, int BH, int N,
    int causal, float scale) {
    constexpr int KS = D / 4, MB = D / 16;
    __shared__ __attribute__((aligned(16))) uint16_t KV0[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t KV1[2][kTile * D];
    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int q0w = tile * kTile + 16 * wave;
    const int qrow = q0w + c16;

    float qf[KS];
    ld_row_perm<D>(make_rsrc(Q + hoff, (uint32_t)N * (2 * D)), qrow, g, qf);

    const KeyRange kr = key_range(tile, N, 0, causal);
    const int nkv = kr.nkv, nplain = kr.nplain;
    const float lg = kLog2e;
    float mrun = -INFINITY, lrun = 0.f;  // scaled running maximum; this lane's share of l
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    TileDma<D> dma;
    dma.init(lane, wave);
    dma.load(K + hoff, KV0[0], 0, N);
    dma.load(V + hoff, KV0[1], 0, N);
    wait_vm_lgkm0<0>();
    __syncthreads();

    auto step = [&](auto masked, int kt, const uint16_t* Kc, const uint16_t* Vc, uint16_t* Kn,
                    uint16_t* Vn) {
        constexpr bool MASK = decltype(masked)::value;
        if (kt + 1 < nkv) {
            dma.load(K + hoff, Kn, (kt + 1) * kTile, N);
            dma.load(V + hoff, Vn, (kt + 1) * kTile, N);
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x4 s[4];
        float tmax = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            s[kb] = block_dot<D>(Kc, 16 * kb, qf, c16, g);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float v = scale * s[kb][i];
                if constexpr (MASK) {
                    const int key = kt * kTile + 16 * kb + 4 * g + i;
                    v = (key < N && (!causal || key <= qrow)) ? v : -INFINITY;
                }
                s[kb][i] = v;
                tmax = fmaxf(tmax, v);
            }
        }
        const float mnew = fmaxf(mrun, xor_max(tmax));
        // a row that has seen no key yet keeps m = -inf; its factors are 1, 0
        const float corr = mnew == -INFINITY ? 1.f : fexp2((mrun - mnew) * lg);
        const float msub = mnew == -INFINITY ? 0.f : mnew;
        mrun = mnew;
        float lsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = fexp2((s[kb][i] - msub) * lg);
                s[kb][i] = p;
                lsum += p;
            }
        lrun = lrun * corr + lsum;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[mb] *= corr;
        tr_accumulate<D>(Vc, s, acc, c16, g);
        wait_vm_lgkm0<0>();
        __syncthreads();
    };
    const std::false_type plain;
    const std::true_type masked;
    int kt = 0;
    for (; kt < nplain; ++kt) {
        if (kt & 1) step(plain, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }
    for (; kt < nkv; ++kt) {
        if (kt & 1) step(masked, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else step(masked, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }

    const float l = xor_sum(lrun);
    if (qrow < N) {
        const float inv = 1.f / l;
        float* orow = O32 + hoff + (size_t)qrow * D;
        uint16_t* brow = O + hoff + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            f32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = acc[mb][i] / l;
            *reinterpret_cast<f32x4*>(orow + 16 * mb + 4 * g) = o;
            st_bf16x4(brow + 16 * mb + 4 * g, o[0], o[1], o[2], o[3]);
        }
        if (g == 0) {
            const size_t r = (size_t)bh * N + qrow;
            LSE[r] = mrun + logf(l);
            Mrow[r] = mrun;
            Linv[r] = inv;
        }
    }
}

// ------------------------------------------------------- query-major pass
template <int D>
__global__ __launch_bounds__(kThreads, 2) void f32_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ O32, const float* __restrict__ Mrow,
    const float* __restrict__ Linv, float* __restrict__ TS, uint16_t* __restrict__ dQ, int BH,
    int N, int causal, float scale) {
    constexpr int KS = D / 4, MB = D / 16;
    __shared__ __attribute__((aligned(16))) uint16_t KV0[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t KV1[2][kTile * D];
    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + 16 * wave + c16;
    const bool qok = qrow < N;

    const uint32_t tb = (uint32_t)N * (2 * D);
    float qf[KS], uf[KS];
    ld_row_perm<D>(make_rsrc(Q + hoff, tb), qrow, g, qf);
    ld_row_perm<D>(make_rsrc(dO + hoff, tb), qrow, g, uf);
    // D_i = sum_d dO_id O32_id (the saved FP32 output), this lane's d subset
    // then the other three lanes of the query.
    float dpart = 0.f;
    if (qok) {
        const float* orow = O32 + hoff + (size_t)qrow * D;
#pragma unroll
        for (int h = 0; h < D / 64; ++h)
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const f32x4 o = *reinterpret_cast<const f32x4*>(orow + 64 * h + 16 * g + 4 * p);
#pragma unroll
                for (int e = 0; e < 4; ++e) dpart = fmaf(uf[16 * h + 4 * p + e], o[e], dpart);
            }
    }
    const float Di = xor_sum(dpart);
    const size_t srow = (size_t)bh * N + qrow;
    const float mi = qok ? Mrow[srow] : INFINITY;  // rows beyond N: P = 0
    const float li = qok ? Linv[srow] : 0.f;
    const float lg = kLog2e;

    const KeyRange kr = key_range(tile, N, 0, causal);
    const int nkv = kr.nkv, nplain = kr.nplain;
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    TileDma<D> dma;
    dma.init(lane, wave);
    wait_vm_lgkm0<0>();
    dma.load(K + hoff, KV0[0], 0, N);
    dma.load(V + hoff, KV0[1], 0, N);
    wait_vm_lgkm0<0>();
    __syncthreads();

    auto step = [&](auto masked, int kt, const uint16_t* Kc, const uint16_t* Vc, uint16_t* Kn,
                    uint16_t* Vn) {
        constexpr bool MASK = decltype(masked)::value;
        if (kt + 1 < nkv) {
            dma.load(K + hoff, Kn, (kt + 1) * kTile, N);
            dma.load(V + hoff, Vn, (kt + 1) * kTile, N);
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x4 ds[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const f32x4 s = block_dot<D>(Kc, 16 * kb, qf, c16, g);
            const f32x4 dp = block_dot<D>(Vc, 16 * kb, uf, c16, g);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float p = fexp2((scale * s[i] - mi) * lg) * li;
                if constexpr (MASK) {
                    const int key = kt * kTile + 16 * kb + 4 * g + i;
                    p = (key < N && (!causal || key <= qrow)) ? p : 0.f;
                }
                ds[kb][i] = p * (dp[i] - Di);
                if constexpr (MASK) ds[kb][i] = p != 0.f ? ds[kb][i] : 0.f;
            }
        }
        tr_accumulate<D>(Kc, ds, acc, c16, g);
        wait_vm_lgkm0<0>();
        __syncthreads();
    };
    const std::false_type plain;
    const std::true_type masked;
    int kt = 0;
    for (; kt < nplain; ++kt) {
        if (kt & 1) step(plain, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else step(plain, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }
    for (; kt < nkv; ++kt) {
        if (kt & 1) step(masked, kt, KV1[0], KV1[1], KV0[0], KV0[1]);
        else step(masked, kt, KV0[0], KV0[1], KV1[0], KV1[1]);
    }

    if (qok) {
        uint16_t* drow = dQ + hoff + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            st_bf16x4(drow + 16 * mb + 4 * g, scale * acc[mb][0], scale * acc[mb][1],
                      scale * acc[mb][2], scale * acc[mb][3]);
    }
    // the tile's statistics for the key-major pass
    if (g == 0) {
        float* ts = TS + ((size_t)bh * T + tile) * kF32Stat + 16 * wave + c16;
        ts[0] = mi;
        ts[kTile] = li;
        ts[2 * kTile] = qok ? Di : 0.f;
    }
}

// --------------------------------------------------------- key-major pass
template <int D>
__global__ __launch_bounds__(kThreads, 2) void f32_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ TS, uint16_t* __restrict__ dK, uint16_t* __restrict__ dV, int BH,
    int N, int causal, float scale) {
    constexpr int KS = D / 4, MB = D / 16;
    __shared__ __attribute__((aligned(16))) uint16_t QU0[2][kTile * D];
    __shared__ __attribute__((aligned(16))) uint16_t QU1[2][kTile * D];
    __shared__ __attribute__((aligned(16))) float ST0[kF32Stat];
    __shared__ __attribute__((aligned(16))) float ST1[kF32Stat];
    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, false, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int krow = tile * kTile + 16 * wave + c16;

    const uint32_t tb = (uint32_t)N * (2 * D);
    float kf[KS], vf[KS];
    ld_row_perm<D>(make_rsrc(K + hoff, tb), krow, g, kf);
    ld_row_perm<D>(make_rsrc(V + hoff, tb), krow, g, vf);
    const float lg = kLog2e;
    const float* tsh = TS + (size_t)bh * T * kF32Stat;

    f32x4 accV[MB], accK[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        accV[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
        accK[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int qt0 = causal ? tile : 0;  // the diagonal tile first, masked

    TileDma<D> dma;
    dma.init(lane, wave);
    // Query tile qt's Q and dO tiles and its statistics block (waves 0..2 each
    // move one 256-byte third of it with a 4-byte LDS DMA), issued through the
    // vector-memory path the closing vmcnt(0) waits for: no load in the loop
    // is visible to the compiler's own wait counting.
    auto fill = [&](int qt, uint16_t (*QU)[kTile * D], float* ST) {
        dma.load(Q + hoff, QU[0], qt * kTile, N);
        dma.load(dO + hoff, QU[1], qt * kTile, N);
        if (wave < 3)
            lds_dma4(buf_desc(tsh + (size_t)qt * kF32Stat + wave * kTile, kTile * 4),
                     lds_addr(ST + wave * kTile), (uint32_t)lane * 4u);
    };
    wait_vm_lgkm0<0>();
    fill(qt0 < T ? qt0 : 0, QU0, ST0);
    wait_vm_lgkm0<0>();
    __syncthreads();

    auto step = [&](auto masked, int qt, uint16_t (*QUc)[kTile * D], const float* st,
                    uint16_t (*QUn)[kTile * D], float* STn) {
        constexpr bool MASK = decltype(masked)::value;
        const uint16_t* Qc = QUc[0];
        const uint16_t* Uc = QUc[1];
        if (qt + 1 < T) fill(qt + 1, QUn, STn);
        __builtin_amdgcn_sched_barrier(0);
        f32x4 p[4], ds[4];
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) {
            const f32x4 mq = *reinterpret_cast<const f32x4*>(st + 16 * qb + 4 * g);
            const f32x4 lq = *reinterpret_cast<const f32x4*>(st + kTile + 16 * qb + 4 * g);
            const f32x4 dq = *reinterpret_cast<const f32x4*>(st + 2 * kTile + 16 * qb + 4 * g);
            const f32x4 s = block_dot<D>(Qc, 16 * qb, kf, c16, g);
            const f32x4 dp = block_dot<D>(Uc, 16 * qb, vf, c16, g);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float pv = fexp2((scale * s[i] - mq[i]) * lg) * lq[i];
                if constexpr (MASK) {
                    const int query = qt * kTile + 16 * qb + 4 * g + i;
                    pv = (!causal || krow <= query) ? pv : 0.f;
                }
                p[qb][i] = pv;
                ds[qb][i] = pv * (dp[i] - dq[i]);
                if constexpr (MASK) ds[qb][i] = pv != 0.f ? ds[qb][i] : 0.f;
            }
        }
        tr_accumulate<D>(Uc, p, accV, c16, g);
        tr_accumulate<D>(Qc, ds, accK, c16, g);
        wait_vm_lgkm0<0>();
        __syncthreads();
    };
    const std::false_type plain;
    const std::true_type masked;
    int qt = qt0;
    // The first tile is staged in slot 0 whatever its index: slots alternate
    // with the step count from qt0.
    if (causal && qt < T) {
        step(masked, qt, QU0, ST0, QU1, ST1);
        ++qt;
    }
    for (; qt < T; ++qt) {
        if ((qt - qt0) & 1) step(plain, qt, QU1, ST1, QU0, ST0);
        else step(plain, qt, QU0, ST0, QU1, ST1);
    }

    if (krow < N) {
        uint16_t* vrow = dV + hoff + (size_t)krow * D;
        uint16_t* krw = dK + hoff + (size_t)krow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            st_bf16x4(vrow + 16 * mb + 4 * g, accV[mb][0], accV[mb][1], accV[mb][2], accV[mb][3]);
            st_bf16x4(krw + 16 * mb + 4 * g, scale * accK[mb][0], scale * accK[mb][1],
                      scale * accK[mb][2], scale * accK[mb][3]);
        }
    }
}

}  // namespace

hipError_t launch_f32_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, float* O32,
                          uint16_t* O, float* LSE, float* Mrow, float* Linv, const Shape& s,
                          hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    if (s.d == 64)
        launch_kernel(f32_fwd_kernel<64>, grid, block, st, Q, K, V, O32, O, LSE, Mrow, Linv, s.BH,
                      s.N, s.causal, s.scale);
    else
        launch_kernel(f32_fwd_kernel<128>, grid, block, st, Q, K, V, O32, O, LSE, Mrow, Linv, s.BH,
                      s.N, s.causal, s.scale);
    return hipGetLastError();
}

hipError_t launch_f32_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, const float* O32, const float* Mrow,
                         const float* Linv, float* TS, uint16_t* dQ, const Shape& s,
                         hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    if (s.d == 64)
        launch_kernel(f32_dq_kernel<64>, grid, block, st, Q, K, V, dO, O32, Mrow, Linv, TS, dQ,
                      s.BH, s.N, s.causal, s.scale);
    else
        launch_kernel(f32_dq_kernel<128>, grid, block, st, Q, K, V, dO, O32, Mrow, Linv, TS, dQ,
                      s.BH, s.N, s.causal, s.scale);
    return hipGetLastError();
}

hipError_t launch_f32_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* TS, uint16_t* dK, uint16_t* dV,
                           const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    if (s.d == 64)
        launch_kernel(f32_dkdv_kernel<64>, grid, block, st, Q, K, V, dO, TS, dK, dV, s.BH, s.N,
                      s.causal, s.scale);
    else
        launch_kernel(f32_dkdv_kernel<128>, grid, block, st, Q, K, V, dO, TS, dK, dV, s.BH, s.N,
                      s.causal, s.scale);
    return hipGetLastError();
}

}  // namespace gpa
