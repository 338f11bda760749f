// FP32 attention baseline: BF16 inputs and outputs, all arithmetic in FP32
// SIMT (no matrix cores, no BF16 intermediates).  This is the accuracy class
// of the paper's "FP32 attention" (appendix on comparison methods; the fused
// variant keeps an FP32 output for the backward's row statistic).  It is the
// yardstick of the "within 2x of FP32 attention" accuracy criterion, not a
// tuned kernel.
//
// Each row (query or key) is handled by D/32 threads of 32 channels each; a
// workgroup covers 64 rows and streams the other operand through LDS as FP32.
#include "gpa_device.h"
#include "gpa_launch.h"

namespace gpa {
namespace {

__device__ __forceinline__ float ld_bf16(const uint16_t* p) {
    return __uint_as_float(((uint32_t)*p) << 16);
}

template <int TPR>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
    for (int off = TPR / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void f32_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ O32, uint16_t* __restrict__ O,
    float* __restrict__ LSE, int BH, int N, int causal, float scale) {
    constexpr int TPR = D / 32, NT = 64 * TPR;
    __shared__ float Kf[64][D + 1];
    __shared__ float Vf[64][D + 1];
    const int T = (N + 63) / 64;
    const int bh = blockIdx.x / T, tile = blockIdx.x - (blockIdx.x / T) * T;
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, rl = tid / TPR, part = tid - rl * TPR;
    const int qrow = tile * 64 + rl;
    const bool qok = qrow < N;
    float q[32], o[32];
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        q[c] = qok ? ld_bf16(Q + hoff + (size_t)qrow * D + part * 32 + c) : 0.f;
        o[c] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int kv_end = causal ? min(N, (tile + 1) * 64) : N;
    for (int k0 = 0; k0 < kv_end; k0 += 64) {
        __syncthreads();
        for (int idx = tid; idx < 64 * D; idx += NT) {
            const int r = idx / D, col = idx - (idx / D) * D, row = k0 + r;
            Kf[r][col] = row < N ? ld_bf16(K + hoff + (size_t)row * D + col) : 0.f;
            Vf[r][col] = row < N ? ld_bf16(V + hoff + (size_t)row * D + col) : 0.f;
        }
        __syncthreads();
        const int jn = min(64, kv_end - k0);
        for (int j = 0; j < jn; ++j) {
            float sd = 0.f;
#pragma unroll
            for (int c = 0; c < 32; ++c) sd = fmaf(q[c], Kf[j][part * 32 + c], sd);
            sd = group_sum<TPR>(sd);
            const int key = k0 + j;
            if (!causal || key <= qrow) {
                const float sv = scale * sd;
                if (sv > m) {
                    const float corr = expf(m - sv);
                    l *= corr;
#pragma unroll
                    for (int c = 0; c < 32; ++c) o[c] *= corr;
                    m = sv;
                }
                const float p = expf(sv - m);
                l += p;
#pragma unroll
                for (int c = 0; c < 32; ++c) o[c] = fmaf(p, Vf[j][part * 32 + c], o[c]);
            }
        }
    }
    if (qok) {
#pragma unroll
        for (int c = 0; c < 32; ++c) {
            const float v = o[c] / l;
            O32[hoff + (size_t)qrow * D + part * 32 + c] = v;
            O[hoff + (size_t)qrow * D + part * 32 + c] = bf16_bits(v);
        }
        if (part == 0) LSE[(size_t)bh * N + qrow] = m + logf(l);
    }
}

template <int D>
__global__ __launch_bounds__(256) void f32_pre_kernel(const float* __restrict__ O32,
                                                      const uint16_t* __restrict__ dO,
                                                      float* __restrict__ Drow, int rows) {
    const int row = blockIdx.x * 256 + threadIdx.x;
    if (row >= rows) return;
    float acc = 0.f;
    for (int c = 0; c < D; ++c)
        acc = fmaf(ld_bf16(dO + (size_t)row * D + c), O32[(size_t)row * D + c], acc);
    Drow[row] = acc;
}

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void f32_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow, uint16_t* __restrict__ dQ,
    int BH, int N, int causal, float scale) {
    constexpr int TPR = D / 32, NT = 64 * TPR;
    __shared__ float Kf[64][D + 1];
    __shared__ float Vf[64][D + 1];
    const int T = (N + 63) / 64;
    const int bh = blockIdx.x / T, tile = blockIdx.x - (blockIdx.x / T) * T;
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, rl = tid / TPR, part = tid - rl * TPR;
    const int qrow = tile * 64 + rl;
    const bool qok = qrow < N;
    float q[32], u[32], dq[32];
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        q[c] = qok ? ld_bf16(Q + hoff + (size_t)qrow * D + part * 32 + c) : 0.f;
        u[c] = qok ? ld_bf16(dO + hoff + (size_t)qrow * D + part * 32 + c) : 0.f;
        dq[c] = 0.f;
    }
    const float lse = qok ? LSE[(size_t)bh * N + qrow] : 0.f;
    const float Di = qok ? Drow[(size_t)bh * N + qrow] : 0.f;
    const int kv_end = causal ? min(N, (tile + 1) * 64) : N;
    for (int k0 = 0; k0 < kv_end; k0 += 64) {
        __syncthreads();
        for (int idx = tid; idx < 64 * D; idx += NT) {
            const int r = idx / D, col = idx - (idx / D) * D, row = k0 + r;
            Kf[r][col] = row < N ? ld_bf16(K + hoff + (size_t)row * D + col) : 0.f;
            Vf[r][col] = row < N ? ld_bf16(V + hoff + (size_t)row * D + col) : 0.f;
        }
        __syncthreads();
        const int jn = min(64, kv_end - k0);
        for (int j = 0; j < jn; ++j) {
            float sd = 0.f, ud = 0.f;
#pragma unroll
            for (int c = 0; c < 32; ++c) {
                sd = fmaf(q[c], Kf[j][part * 32 + c], sd);
                ud = fmaf(u[c], Vf[j][part * 32 + c], ud);
            }
            sd = group_sum<TPR>(sd);
            ud = group_sum<TPR>(ud);
            const int key = k0 + j;
            if (qok && (!causal || key <= qrow)) {
                const float p = expf(scale * sd - lse);
                const float ds = p * (ud - Di);
#pragma unroll
                for (int c = 0; c < 32; ++c) dq[c] = fmaf(ds, Kf[j][part * 32 + c], dq[c]);
            }
        }
    }
    if (qok) {
#pragma unroll
        for (int c = 0; c < 32; ++c)
            dQ[hoff + (size_t)qrow * D + part * 32 + c] = bf16_bits(scale * dq[c]);
    }
}

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void f32_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ LSE, const float* __restrict__ Drow, uint16_t* __restrict__ dK,
    uint16_t* __restrict__ dV, int BH, int N, int causal, float scale) {
    constexpr int TPR = D / 32, NT = 64 * TPR;
    __shared__ float Qf[64][D + 1];
    __shared__ float Uf[64][D + 1];
    __shared__ float Ls[64];
    __shared__ float Dsh[64];
    const int T = (N + 63) / 64;
    const int bh = blockIdx.x / T, tile = blockIdx.x - (blockIdx.x / T) * T;
    const size_t hoff = (size_t)bh * N * D;
    const int tid = threadIdx.x, rl = tid / TPR, part = tid - rl * TPR;
    const int krow = tile * 64 + rl;
    const bool kok = krow < N;
    float k[32], v[32], dk[32], dv[32];
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        k[c] = kok ? ld_bf16(K + hoff + (size_t)krow * D + part * 32 + c) : 0.f;
        v[c] = kok ? ld_bf16(V + hoff + (size_t)krow * D + part * 32 + c) : 0.f;
        dk[c] = 0.f;
        dv[c] = 0.f;
    }
    const int q_begin = causal ? tile * 64 : 0;
    for (int q0 = q_begin; q0 < N; q0 += 64) {
        __syncthreads();
        for (int idx = tid; idx < 64 * D; idx += NT) {
            const int r = idx / D, col = idx - (idx / D) * D, row = q0 + r;
            Qf[r][col] = row < N ? ld_bf16(Q + hoff + (size_t)row * D + col) : 0.f;
            Uf[r][col] = row < N ? ld_bf16(dO + hoff + (size_t)row * D + col) : 0.f;
        }
        if (tid < 64) {
            const int row = q0 + tid;
            Ls[tid] = row < N ? LSE[(size_t)bh * N + row] : 0.f;
            Dsh[tid] = row < N ? Drow[(size_t)bh * N + row] : 0.f;
        }
        __syncthreads();
        const int in = min(64, N - q0);
        for (int i = 0; i < in; ++i) {
            float sd = 0.f, ud = 0.f;
#pragma unroll
            for (int c = 0; c < 32; ++c) {
                sd = fmaf(Qf[i][part * 32 + c], k[c], sd);
                ud = fmaf(Uf[i][part * 32 + c], v[c], ud);
            }
            sd = group_sum<TPR>(sd);
            ud = group_sum<TPR>(ud);
            const int query = q0 + i;
            if (kok && (!causal || krow <= query)) {
                const float p = expf(scale * sd - Ls[i]);
                const float ds = p * (ud - Dsh[i]);
#pragma unroll
                for (int c = 0; c < 32; ++c) {
                    dk[c] = fmaf(ds, Qf[i][part * 32 + c], dk[c]);
                    dv[c] = fmaf(p, Uf[i][part * 32 + c], dv[c]);
                }
            }
        }
    }
    if (kok) {
#pragma unroll
        for (int c = 0; c < 32; ++c) {
            dK[hoff + (size_t)krow * D + part * 32 + c] = bf16_bits(scale * dk[c]);
            dV[hoff + (size_t)krow * D + part * 32 + c] = bf16_bits(dv[c]);
        }
    }
}

}  // namespace

#define GPA_D_DISPATCH(KERNEL, GRID, BLOCK_OF_D, ...)                                 \
    do {                                                                              \
        if (s.d == 64)                                                                \
            KERNEL<64><<<(GRID), BLOCK_OF_D(64), 0, st>>>(__VA_ARGS__);               \
        else                                                                          \
            KERNEL<128><<<(GRID), BLOCK_OF_D(128), 0, st>>>(__VA_ARGS__);             \
    } while (0)
#define GPA_ROWS_BLOCK(DD) (64 * ((DD) / 32))

hipError_t launch_f32_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, float* O32,
                          uint16_t* O, float* LSE, const Shape& s, hipStream_t st) {
    const unsigned grid = (unsigned)(s.BH * ((s.N + 63) / 64));
    GPA_D_DISPATCH(f32_fwd_kernel, grid, GPA_ROWS_BLOCK, Q, K, V, O32, O, LSE, s.BH, s.N,
                   s.causal, s.scale);
    return hipGetLastError();
}

hipError_t launch_f32_pre(const float* O32, const uint16_t* dO, float* Drow, const Shape& s,
                          hipStream_t st) {
    const int rows = s.BH * s.N;
    const unsigned grid = (unsigned)((rows + 255) / 256);
#define GPA_256(DD) 256
    GPA_D_DISPATCH(f32_pre_kernel, grid, GPA_256, O32, dO, Drow, rows);
#undef GPA_256
    return hipGetLastError();
}

hipError_t launch_f32_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, const float* LSE, const float* Drow, uint16_t* dQ,
                         const Shape& s, hipStream_t st) {
    const unsigned grid = (unsigned)(s.BH * ((s.N + 63) / 64));
    GPA_D_DISPATCH(f32_dq_kernel, grid, GPA_ROWS_BLOCK, Q, K, V, dO, LSE, Drow, dQ, s.BH, s.N,
                   s.causal, s.scale);
    return hipGetLastError();
}

hipError_t launch_f32_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* LSE, const float* Drow,
                           uint16_t* dK, uint16_t* dV, const Shape& s, hipStream_t st) {
    const unsigned grid = (unsigned)(s.BH * ((s.N + 63) / 64));
    GPA_D_DISPATCH(f32_dkdv_kernel, grid, GPA_ROWS_BLOCK, Q, K, V, dO, LSE, Drow, dK, dV, s.BH,
                   s.N, s.causal, s.scale);
    return hipGetLastError();
}

}  // namespace gpa
