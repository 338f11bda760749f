// Host-side launchers of the libgpa kernels (internal; the public interface is
// include/gpa.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

namespace gpa {

// Events of the launch being timed (both null unless the ABI layer's kernel
// timing is on).  Per host thread.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
LaunchEvents& launch_events();

// Launch `kernel` on `st` with the arguments converted to its parameter types
// (their count must match).  While kernel timing is on, the launch goes
// through hipExtLaunchKernel, which records the events when the kernel starts
// and when it ends, so the elapsed time between them is the kernel's own
// duration (events recorded around the launch would add the dispatch gap);
// otherwise it is a plain hipLaunchKernel.  Errors are left for
// hipGetLastError.
template <typename... Formals, typename... Actuals>
inline void launch_kernel(void (*kernel)(Formals...), dim3 grid, dim3 block, hipStream_t st,
                          Actuals... actuals) {
    static_assert(sizeof...(Formals) == sizeof...(Actuals), "kernel argument count");
    std::tuple<Formals...> args{actuals...};
    std::apply(
        [&](auto&... a) {
            void* ptrs[] = {static_cast<void*>(&a)...};
            const LaunchEvents& e = launch_events();
            if (e.start != nullptr || e.stop != nullptr)
                (void)hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs,
                                         0, st, e.start, e.stop, 0);
            else
                (void)hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, 0,
                                      st);
        },
        args);
}

struct Shape {
    int BH;        // batch * query heads (packed sequences: sequences * query heads)
    int N;         // sequence length (packed sequences: the longest one)
    int d;         // head dimension (64 or 128)
    int causal;    // 1: key j visible to query i iff j <= i
    float scale;   // attention scale alpha
    int G;         // query heads per key/value head (1: multi-head attention);
                   // query head bh reads key/value head bh / G
    // Packed variable-length sequences (nullptr: dense [B, H, N, d] batches).
    // Query-side tensors are [H, total, d] and key-side ones [H, total_k, d];
    // sequence s holds queries [cu[s], cu[s + 1]) and keys
    // [cu_k[s], cu_k[s + 1]), and problem bh = s * Hq + h is head h of
    // sequence s.  N is then the longest query run and Nk the longest key run.
    const int* cu = nullptr;    // device, nseq + 1 query offsets
    int Hq = 1;                 // query heads
    int total = 0;              // query tokens in the packed tensors
    const int* cu_k = nullptr;  // device, nseq + 1 key offsets
    int total_k = 0;            // key tokens in the packed tensors
    int Nk = 0;                 // longest key run (dense: N)
};

// Kernel ids for timing (gpa_profile_*).
enum KernelId {
    kKFwd = 0,
    kKBwdDq = 1,
    kKBwdDkdv = 2,
    kKF32Fwd = 3,
    kKF32Dq = 4,
    kKF32Dkdv = 5,
    kKGroupSum = 6,
    kKBwdPre = 7,
    kKBwdFused = 8,
    kKBwdFinal = 9,
    kKBwdCorr = 10,
    kNumKernels = 11
};

// fma_forward selects the historical exponent rounding (diagnostic only).
hipError_t launch_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, uint16_t* O,
                      float* LSE, const Shape& s, hipStream_t st, bool fma_forward = false);

// Query-major pass: writes D = rowsum(dO * O) and dQ; in the gproj modes also
// rho, m, lambda (zero in plain mode); in gproj mode also Z = BF16(-lambda Q)
// ([BH, N, d], BF16).  TS ([BH, T, 2, 64] FP32, T = tiles of 64 rows)
// receives per tile LSE * log2(e) (+inf beyond N) and D (0 beyond N) for the
// key pass.
hipError_t launch_bwd_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* O, const uint16_t* dO, const float* LSE, float* Drow,
                         float* TS, uint16_t* dQ, float* rho, float* msum, float* lambda,
                         uint16_t* Z, int mode, const Shape& s, hipStream_t st);

// Key-major pass: dV = r^T dO, dK = t^T Q (minus r^T Z in gproj mode).  With
// G == 1 it writes BF16 dK, dV; with G > 1 every query head writes its FP32
// contributions (dKp = t^T Q - r^T Z unscaled, dVp = r^T dO; [BH, N, d]) and
// launch_bwd_group_sum adds them per key/value head.
hipError_t launch_bwd_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* TS, const uint16_t* Z,
                           uint16_t* dK, uint16_t* dV, float* dKp, float* dVp, int mode,
                           const Shape& s, hipStream_t st);

// FP32 accumulators of the atomic schedule ([BH, N, d] for A, B and dK^acc,
// [BH, N] for rho and m); B, rho, m are null in plain mode, dKacc outside
// gproj mode.
struct AtomicAcc {
    float* A = nullptr;
    float* B = nullptr;
    float* rho = nullptr;
    float* m = nullptr;
    float* dKacc = nullptr;
};

// Algorithm 1's schedule with atomics (dense multi-head): launch_bwd_pre
// writes the per-tile statistics TS ([BH, T, 2, 64], as the query-major pass
// does, same D bits) and zeroes the accumulators; launch_bwd_fused runs the
// single key-major pass: dV, and dK (plain, gproj_q: the plain key pass's
// arithmetic) or the FP32 dK^acc (gproj), with t K (and in the GProj modes
// r K, rho, m) added by atomics; launch_bwd_dq_finalize writes
// dQ = BF16(scale * A) (plain); launch_bwd_gproj_finalize forms lambda, dQ
// and, with Zneg, -z = BF16(-lambda Q); launch_bwd_dk_corr is the gproj
// correction pass that writes dK.
hipError_t launch_bwd_pre(const uint16_t* O, const uint16_t* dO, const float* LSE, float* TS,
                          const AtomicAcc& a, const Shape& s, hipStream_t st);
hipError_t launch_bwd_fused(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            const uint16_t* dO, const float* TS, uint16_t* dK, uint16_t* dV,
                            const AtomicAcc& a, int mode, const Shape& s, hipStream_t st);
hipError_t launch_bwd_dq_finalize(const float* dQacc, uint16_t* dQ, const Shape& s,
                                  hipStream_t st);
hipError_t launch_bwd_gproj_finalize(const AtomicAcc& a, const uint16_t* Q, uint16_t* dQ,
                                     uint16_t* Zneg, float* lam, const Shape& s, hipStream_t st);
hipError_t launch_bwd_dk_corr(const uint16_t* Q, const uint16_t* K, const float* TS,
                              const uint16_t* Zneg, const float* dKacc, uint16_t* dK,
                              const Shape& s, hipStream_t st);

// dK = BF16(scale * sum_g dKp), dV = BF16(sum_g dVp) over the G query heads of
// each key/value head, in head order.
hipError_t launch_bwd_group_sum(const float* dKp, const float* dVp, uint16_t* dK, uint16_t* dV,
                                const Shape& s, hipStream_t st);

// Fused FP32 baseline.  The forward writes O (BF16), LSE and, in the
// workspace, the FP32 output O32 and the scaled row maximum and inverse
// normaliser per row ([BH, N] each).  The query-major pass forms D =
// rowsum(dO O32), writes dQ and the per-tile statistics TS ([BH, T, 3, 64]:
// row maximum, inverse normaliser, D; +inf, 0, 0 beyond N) that the
// key-major pass stages with each query tile.
hipError_t launch_f32_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, float* O32,
                          uint16_t* O, float* LSE, float* Mrow, float* Linv, const Shape& s,
                          hipStream_t st);
hipError_t launch_f32_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, const float* O32, const float* Mrow,
                         const float* Linv, float* TS, uint16_t* dQ, const Shape& s,
                         hipStream_t st);
hipError_t launch_f32_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* TS, uint16_t* dK, uint16_t* dV,
                           const Shape& s, hipStream_t st);

}  // namespace gpa
