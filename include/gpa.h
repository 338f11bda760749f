/*
 * gpa.h -- BF16 attention with the GProj gradient correction, for AMD MI355X
 * (gfx950).  C ABI of libgpa.so.
 *
 * The method is "GProj" (gauge projection) from "Broken Symmetry in BF16
 * Attention: Why FlashAttention Gradients Blow Up Late in Training":
 *   - the forward is FA3-SBS: the softmax subtracts the unscaled row maximum
 *     with an explicitly rounded FP32 subtraction before scaling (appendix
 *     "Implemented Arithmetic and Rounding", eq. gproj-forward);
 *   - the backward is the native mixed-precision attention backward (BF16
 *     matrix products, FP32 accumulators) with, in the gproj modes, the rank-one
 *     correction that restores the zero row sum of the BF16 score-gradient
 *     operand t after its cast: lambda_i = rho_i / m_i with rho_i = sum_j t_ij
 *     and m_i = sum_j r_ij, r = BF16(P); dQ = alpha (tK - lambda (rK)) and
 *     dK = alpha (t^T Q - r^T BF16(lambda Q))  (Section 4; Algorithm 1; eqs.
 *     gproj-row-mass, gproj-accumulators, gproj-query-implemented,
 *     gproj-key-implemented).
 *
 * Conventions shared by every entry point
 *   Layout   Q, K, V, O, dO, dQ, dK, dV are [B, H, N, d] contiguous, d innermost,
 *            BF16 passed as raw 16-bit patterns (uint16_t).  LSE is FP32 [B, H, N].
 *            The plain entry points are multi-head attention (H query heads =
 *            H key/value heads); the *_gqa ones take grouped-query attention:
 *            Q, O, dO, dQ, LSE have Hq heads, K, V, dK, dV have Hkv heads,
 *            Hq a multiple of Hkv, and query head h reads key/value head
 *            h / (Hq / Hkv) (consecutive query heads share one).
 *   Shapes   B, H, N >= 1; d in {64, 128}; B*H*N*d < 2^31.
 *   Causal   causal != 0 means query i attends to keys j <= i (square N x N).
 *   Scale    alpha (the attention scale), finite and > 0; usually 1/sqrt(d).
 *   Pointers device pointers, 16-byte aligned.  Outputs must not overlap any
 *            input, any other output or the workspace.
 *   Stream   a hipStream_t passed as void* (NULL = the null stream).  All work
 *            is enqueued on it asynchronously; the library never synchronises,
 *            never allocates or frees device memory, and fully overwrites every
 *            output.  Calls only enqueue kernels, so they can be captured into
 *            HIP graphs.
 *   Errors   arguments are validated before anything is launched; on error no
 *            work is enqueued and nothing is written.  GPA_EHIP reports a launch
 *            failure (text in gpa_last_error(), per thread).  No C++ exception
 *            crosses this interface.
 */
#ifndef GPA_H
#define GPA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GPA_OK = 0,
    GPA_EINVAL = 1,      /* null/misaligned pointer, bad size, scale, mode or aliasing */
    GPA_ENOTSUP = 2,     /* head dimension other than 64 or 128 */
    GPA_EWORKSPACE = 3,  /* workspace null or smaller than required */
    GPA_EHIP = 4         /* a HIP launch failed */
} gpa_status;

typedef enum {
    GPA_MODE_PLAIN = 0,   /* FA3-SBS backward: no correction */
    GPA_MODE_GPROJ_Q = 1, /* query correction only: dQ projected, dK and dV as plain */
    GPA_MODE_GPROJ = 2    /* query and key corrections: dQ as gproj_q, dK projected */
} gpa_mode;

/* Library version string, e.g. "gpa 0.1.0 gfx950". */
const char* gpa_version(void);

/* Text of a status code (static storage). */
const char* gpa_status_str(gpa_status s);

/* Message of the last error reported on the calling thread ("" if none). */
const char* gpa_last_error(void);

/*
 * Forward (FA3-SBS; eq. gproj-forward; Algorithm 1 input state).
 *   x = Q K^T (unscaled logits, BF16 products, FP32 accumulation), masked;
 *   z = exp2( fl32[ fl32(x - xmax) * fl32(scale*log2 e) ] ) with xmax the
 *   running row maximum (the same rule rescales the running sums);
 *   l = sum z (FP32), O = BF16( sum BF16(z) V / l ), LSE = scale*xmax + ln l.
 * In : Q, K, V  [B,H,N,d] BF16.
 * Out: O [B,H,N,d] BF16; LSE [B,H,N] FP32, natural log of the scaled scores.
 */
gpa_status gpa_attn_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        uint16_t* O, float* LSE,
                        int64_t B, int64_t H, int64_t N, int64_t d,
                        int causal, float scale, void* stream);

/*
 * Workspace bytes gpa_attn_bwd needs for this shape and mode (> 0 for valid
 * shapes, 0 for invalid arguments).  The caller allocates it; its contents on
 * entry do not matter.  It holds the FP32 row statistics D, rho, m, lambda
 * ([B,H,N] each), a per-64-row-tile copy of log2-scaled LSE and D for the
 * key-major pass, and in gproj mode the BF16 [B,H,N,d] tensor -z = BF16(-lambda q).
 * (The paper's schedule adds a query-shaped FP32 workspace and two FP32 row
 * statistics to the native backward: appendix "Implemented Arithmetic and
 * Rounding", paragraph "Cost".  This two-pass schedule keeps the FP32
 * accumulators A = tK and B = rK in registers, so only the row statistics and
 * z reach memory; gpa_attn_bwd_atomic_workspace_bytes sizes Algorithm 1's
 * schedule with its FP32 accumulators.)
 */
size_t gpa_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d, int mode);

/*
 * Backward (Algorithm 1 with the GProj additions).
 * In : Q, K, V, O, dO [B,H,N,d] BF16; LSE [B,H,N] FP32 -- O and LSE as written
 *      by gpa_attn_fwd with the same causal and scale.
 * Out: dQ, dK, dV [B,H,N,d] BF16.
 *   D_i   = sum_c fl32(dO_ic O_ic)     (Algorithm 1's preprocessing, fused
 *                                        into the query-major pass)
 *   P_ij  = exp(scale x_ij - LSE_i) masked, r = BF16(P),
 *   t_ij  = BF16( fl32[ P_ij (dP_ij - D_i) ] ), dP = dO V^T
 *   dV    = BF16( r^T dO )                                   (every mode)
 *   plain   : dQ = BF16(scale * tK),  dK = BF16(scale * t^T Q)
 *   gproj_q : lambda_i = rho_i / m_i (0 where m_i == 0), rho = rowsum(t),
 *             m = rowsum(r); dQ = BF16( fl32[scale (tK - lambda rK)] );
 *             dK, dV bitwise equal to plain
 *   gproj   : as gproj_q, and dK = BF16( fl32[scale (t^T Q - r^T z)] ),
 *             z_i = BF16(lambda_i q_i), with t^T Q and r^T (-z) added into
 *             one FP32 accumulator; dQ, dV bitwise equal to gproj_q
 * All FP32 accumulations are over BF16 products.  The schedule is
 * deterministic: repeated calls give bitwise identical results.
 * workspace: device buffer of at least gpa_attn_bwd_workspace_bytes(...)
 * bytes, 256-byte aligned.  After the call it holds the FP32 row statistics
 * D, rho, m, lambda at the offsets reported by gpa_bwd_stats_offsets (rho, m
 * and lambda are zero in plain mode).
 */
gpa_status gpa_attn_bwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* O, const float* LSE, const uint16_t* dO,
                        uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                        int64_t B, int64_t H, int64_t N, int64_t d,
                        int causal, float scale, int mode,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, arithmetic and results as
 * gpa_attn_bwd (multi-head only) -- bitwise the same outputs -- but its
 * scratch (the row statistics, the per-tile statistics and z, exactly what
 * gpa_attn_bwd keeps in its workspace) lives in the library's own static
 * device array of gpa_attn_bwd_noalloc_max_bytes() bytes (64 MiB), one per
 * GPU, held until the process ends.  The array of the current device is
 * used: the stream must belong to it.  No call allocates or frees memory;
 * the first call on a device looks up the array's address there
 * (hipGetSymbolAddress).  Nothing in the scratch needs to start at any
 * value: every call writes what it reads.  Every call on one GPU shares the
 * array, so calls that overlap in time on one GPU (concurrent streams,
 * threads) race and give wrong results; serialise them.
 * Errors as gpa_attn_bwd, and GPA_EWORKSPACE (nothing launched) when the
 * shape needs more scratch than the array holds, i.e. when
 * gpa_attn_bwd_workspace_bytes(B, H, N, d, mode) > gpa_attn_bwd_noalloc_max_bytes()
 * (e.g. B*H*N above about 430 000 rows at d = 64 in gproj mode).
 */
size_t gpa_attn_bwd_noalloc_max_bytes(void);
gpa_status gpa_attn_bwd_noalloc(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                                const uint16_t* O, const float* LSE, const uint16_t* dO,
                                uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                                int64_t B, int64_t H, int64_t N, int64_t d,
                                int causal, float scale, int mode, void* stream);

/*
 * The backward with Algorithm 1's own schedule (dense multi-head; arguments as
 * gpa_attn_bwd), for measurement beside the two-pass schedule gpa_attn_bwd
 * uses: one key-major pass in which dK and dV stay with their key tile while
 * the query-side sums are added into FP32 accumulators with device-scope
 * atomics.  Kernels, in stream order:
 *   1. D and the per-tile statistics (bitwise those of gpa_attn_bwd's
 *      query-major pass), accumulators zeroed;
 *   2. the key-major pass (Algorithm 1's first loop): dV, and dK (plain,
 *      gproj_q: bitwise gpa_attn_bwd's) or the FP32 dK^acc = t^T Q (gproj);
 *      A = tK by atomics, and in the GProj modes also B = rK and the row
 *      masses rho = sum t, m = sum r (eq. gproj-row-mass);
 *   3. dQ = BF16(fl32(scale A)) (plain), or lambda = rho/m and
 *      dQ = BF16(fl32[scale (A - lambda B)]) (eq. gproj-query-implemented),
 *      with -z = BF16(-lambda q) in gproj mode;
 *   4. gproj mode only, the second key-major pass (Algorithm 1's correction
 *      loop): r-tilde rebuilt (bitwise the first pass's r), C = r-tilde^T z,
 *      dK = BF16(fl32[scale (dK^acc - C)]) (eq. gproj-key-implemented).
 * dV is bitwise that of gpa_attn_bwd in every mode.  The atomic order varies
 * between runs, so dQ (and through lambda the gproj dK) is not bitwise
 * reproducible: its FP32 sums hold the same terms in another order.
 * workspace: at least gpa_attn_bwd_atomic_workspace_bytes(..., mode) bytes,
 * 256-byte aligned (0 for an invalid shape or mode).  Errors as gpa_attn_bwd.
 */
size_t gpa_attn_bwd_atomic_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d,
                                           int mode);
gpa_status gpa_attn_bwd_atomic(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               const uint16_t* O, const float* LSE, const uint16_t* dO,
                               uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                               int64_t B, int64_t H, int64_t N, int64_t d,
                               int causal, float scale, int mode,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * Byte offsets, inside the backward workspace, of the FP32 [B,H,N] arrays D
 * (preprocess row statistic), rho (row mass of t), m (row mass of r) and
 * lambda = rho/m (Algorithm 1; eq. gproj-row-mass).  Any pointer may be NULL.
 */
gpa_status gpa_bwd_stats_offsets(int64_t B, int64_t H, int64_t N, int64_t d, int mode,
                                 size_t* off_D, size_t* off_rho, size_t* off_m,
                                 size_t* off_lambda);

/*
 * Diagnostic forward, not part of the GProj path: gpa_attn_fwd with the
 * historical exponent rounding r = fma(x, a, -fl32(m a)), z = exp2(r), a =
 * fl32(scale log2 e), m the running row maximum (appendix on the source of the
 * saved-output error, eq. historical-fma), everything else as gpa_attn_fwd.
 * Because r is the rounding error of x a instead of 0 when x = m, a row with a
 * single visible key can return BF16(BF16(z) v / z) != v (eq.
 * historical-one-key).  Multi-head only; same arguments and errors as
 * gpa_attn_fwd.
 */
gpa_status gpa_attn_fwd_fma(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            uint16_t* O, float* LSE,
                            int64_t B, int64_t H, int64_t N, int64_t d,
                            int causal, float scale, void* stream);

/*
 * Grouped-query attention (Section 3.2, eq. row-gradients: key and value
 * gradients also sum over the query heads that share a KV head; appendix
 * "Gauge Projection: Proofs", "Rounding in the implemented key correction":
 * GQA only enlarges the set of query rows contributing to a key).  Same
 * arithmetic as gpa_attn_fwd / gpa_attn_bwd per query head; shapes as in the
 * Layout convention with Hq query and Hkv key/value heads.  In the backward,
 * lambda and z stay per query-head row, and for each key/value head
 *   dV = BF16( sum_h r_h^T dO_h ),
 *   dK = BF16( fl32[ scale * sum_h fl32(t_h^T Q_h - r_h^T z_h) ] )   (gproj;
 *        without the r^T z term in plain and gproj_q),
 * the per-head FP32 terms added in head order (deterministic).  With
 * Hq == Hkv these are exactly gpa_attn_fwd / gpa_attn_bwd.  The workspace
 * (gpa_attn_bwd_gqa_workspace_bytes) begins with the layout gpa_bwd_stats_offsets
 * reports for B, H = Hq.  Errors as for the multi-head entry points, plus
 * GPA_EINVAL when Hq is not a positive multiple of Hkv.
 */
gpa_status gpa_attn_fwd_gqa(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            uint16_t* O, float* LSE,
                            int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d,
                            int causal, float scale, void* stream);

size_t gpa_attn_bwd_gqa_workspace_bytes(int64_t B, int64_t Hq, int64_t Hkv, int64_t N,
                                        int64_t d, int mode);

gpa_status gpa_attn_bwd_gqa(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            const uint16_t* O, const float* LSE, const uint16_t* dO,
                            uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                            int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d,
                            int causal, float scale, int mode,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * Packed variable-length sequences (the paper's kernel supports dense and
 * packed causal layouts, Section 5; its synthetic suite covers packed
 * segments, unequal lengths, singleton and tile-boundary rows, appendix
 * "Synthetic Numerical Suite").  nseq sequences are concatenated along the
 * token axis: sequence s holds queries [cu_seqlens_q[s], cu_seqlens_q[s+1])
 * and keys [cu_seqlens_k[s], cu_seqlens_k[s+1]), and attention never crosses
 * a sequence boundary.  With causal, query i of a sequence with nq queries and
 * nk keys sees key j iff j <= i + (nk - nq): the causal diagonal is aligned
 * at the last query and key (for nq == nk, the usual j <= i).  A query that
 * sees no key (nk == 0, or i < nq - nk under causal) is an empty row: its O
 * and dQ are 0, its LSE is +inf, and its rho, m and lambda are 0 (the
 * Algorithm 1 guard for m = 0).  Each (sequence, query head) with nq == nk is
 * exactly the problem gpa_attn_fwd_gqa / gpa_attn_bwd_gqa solve for one head
 * with N = its length, with the same arithmetic and the same kernels.
 *   Layout     Q, O, dO, dQ [Hq, total_q, d]; K, V, dK, dV [Hkv, total_k, d]
 *              (row t of head h at (h * total + t) * d); LSE and the workspace
 *              row statistics [Hq, total_q].  Grouped-query heads as in the
 *              *_gqa entry points.
 *   Offsets    cu_seqlens_q, cu_seqlens_k: device int32 arrays of nseq + 1
 *              offsets, read on the device: [0] = 0, non-decreasing,
 *              [nseq] = total_q (total_k), and no run longer than
 *              max_seqlen_q (max_seqlen_k), host values that size the grids
 *              and the workspace.  cu_seqlens_k NULL means cu_seqlens_q (then
 *              total_k and max_seqlen_k must equal total_q and max_seqlen_q).
 *              Sequences of length 0 are allowed.  The kernels clamp every
 *              offset to [0, total] and every length to its max_seqlen, so
 *              offsets that break these rules cannot make them touch memory
 *              outside the tensors; rows no sequence covers are then left
 *              unwritten and the results are unspecified.  Both arrays need
 *              4-byte alignment and may not overlap an output.
 *   Shapes     nseq >= 1, 1 <= max_seqlen_q <= total_q,
 *              1 <= max_seqlen_k <= total_k, Hq*total_q*d < 2^31,
 *              Hq*total_k*d < 2^31,
 *              nseq*Hq*ceil(max(max_seqlen_q, max_seqlen_k)/64) < 2^31.
 * The workspace layout begins like gpa_attn_bwd's with [Hq, total_q] row
 * statistics (D, rho, m, lambda at the offsets gpa_bwd_stats_offsets reports
 * for B = 1, H = Hq, N = total_q).  Errors as for the *_gqa entry points.
 */
gpa_status gpa_attn_fwd_varlen(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               uint16_t* O, float* LSE, const int32_t* cu_seqlens_q,
                               const int32_t* cu_seqlens_k, int64_t nseq, int64_t total_q,
                               int64_t total_k, int64_t Hq, int64_t Hkv, int64_t max_seqlen_q,
                               int64_t max_seqlen_k, int64_t d, int causal, float scale,
                               void* stream);

size_t gpa_attn_bwd_varlen_workspace_bytes(int64_t nseq, int64_t total_q, int64_t total_k,
                                           int64_t Hq, int64_t Hkv, int64_t max_seqlen_q,
                                           int64_t max_seqlen_k, int64_t d, int mode);

gpa_status gpa_attn_bwd_varlen(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               const uint16_t* O, const float* LSE, const uint16_t* dO,
                               uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                               const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                               int64_t nseq, int64_t total_q, int64_t total_k, int64_t Hq,
                               int64_t Hkv, int64_t max_seqlen_q, int64_t max_seqlen_k, int64_t d,
                               int causal, float scale, int mode, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * FP32 attention baseline (the accuracy class of the paper's "FP32 attention",
 * appendix on comparison methods: BF16 inputs and outputs, FP32 SIMT
 * arithmetic, no BF16 or reduced-precision matrix products).  One call runs
 * forward and backward:
 * In : Q, K, V, dO [B,H,N,d] BF16.
 * Out: O, dQ, dK, dV [B,H,N,d] BF16 (RNE casts of FP32 results); LSE [B,H,N] FP32.
 * The FP32 output (not its BF16 cast) feeds the backward's D = rowsum(dO O).
 * workspace: at least gpa_fp32_attn_workspace_bytes(...) bytes, 256-byte aligned.
 */
size_t gpa_fp32_attn_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d);
gpa_status gpa_fp32_attn(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, uint16_t* O, float* LSE,
                         uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                         int64_t B, int64_t H, int64_t N, int64_t d,
                         int causal, float scale,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Kernel timing for measurement.  While enabled, every kernel the library
 * launches records a pair of HIP events at its own start and end on its
 * stream (hipExtLaunchKernel's start and stop events).  gpa_profile_read
 * synchronises those events, writes per-kernel totals (milliseconds) and launch
 * counts for kernel ids 0..n-1 (see gpa_kernel_name), clears them, and
 * returns the number of ids.  Not thread-safe and not for calls under stream
 * capture (keep it off while capturing a graph); meant for benchmarks.
 */
void gpa_profile_enable(int on);
int gpa_profile_read(double* total_ms, int64_t* launches, int n);
const char* gpa_kernel_name(int id);

#ifdef __cplusplus
}
#endif

#endif /* GPA_H */
