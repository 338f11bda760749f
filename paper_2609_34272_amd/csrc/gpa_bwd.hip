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
//                  It also forms D_i = rowsum(dO_i * O_i) (FP32) for its rows,
//                  and in gproj mode writes z = BF16(lambda q), once per row.
//   2. bwd_dkdv  : key-major.  A workgroup owns 64 keys and streams the query
//                  tiles (Q, dO and -z); it accumulates dV = r^T dO and, in one
//                  FP32 accumulator, dK^acc - C = t^T Q + r^T (-z), and writes
//                  dK = BF16(fl32[alpha (dK^acc - C)]).  (The paper keeps two
//                  accumulators and subtracts them; one accumulator holds the
//                  same BF16 products summed in another FP32 order.)
// Both passes rebuild P, r and t with identical instructions, so the r and t
// of the key pass equal those of the query pass bitwise, and lambda is divided
// once.  gproj_q runs the GProj query pass and the plain key pass; gproj runs
// both GProj passes.  FP32 accumulators, BF16 operands and the cast points are
// those of the paper; only where lambda becomes available differs.
//
// Work split inside a workgroup (4 waves).  Each wave owns 32 of the
// workgroup's 64 rows (two 16-row MFMA blocks that share every LDS operand
// fragment) and half of each streamed tile; the two waves that own the same
// rows add their partial accumulators through LDS at the end.  The d = 128
// query pass, whose 32-row waves fill the register file (one wave per SIMD),
// runs 8 waves of one 16-row block each instead: two waves per SIMD, each K
// and V fragment feeding one MFMA instead of two.
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

#include <type_traits>

namespace gpa {
namespace {

// Pairwise reduction of per-lane FP32 partials between waves w and w + QG:
// waves QG .. 2 QG - 1 park their values in LDS (lane-contiguous,
// conflict-free), waves 0 .. QG - 1 add them.  `scratch` holds CAP floats;
// the values go through it in rounds of CAP / (64 QG) per lane.  The caller has synchronised the workgroup so
// the buffer is free; on return it is free again only after a barrier.
template <int NV, int CAP, int QG = 2>
__device__ __forceinline__ void pair_reduce(float (&v)[NV], float* scratch, int wave, int lane) {
    constexpr int PER = CAP / (64 * QG);
    static_assert(PER >= 1, "scratch too small");
#pragma unroll
    for (int j0 = 0; j0 < NV; j0 += PER) {
        if (j0) __syncthreads();
        if (wave >= QG) {
            float* p = scratch + (wave - QG) * 64 * PER + lane;
#pragma unroll
            for (int j = j0; j < (j0 + PER < NV ? j0 + PER : NV); ++j) p[(j - j0) * 64] = v[j];
        }
        __syncthreads();
        if (wave < QG) {
            const float* p = scratch + wave * 64 * PER + lane;
#pragma unroll
            for (int j = j0; j < (j0 + PER < NV ? j0 + PER : NV); ++j) v[j] += p[(j - j0) * 64];
        }
    }
}

// --------------------------------------------------------- query-major pass
// P, r, t of one 32-key x 16-query block pair: s[kb], dp[kb] hold keys
// 4g+i of key block kb for this lane's query.  MASK applies the causal and
// tail masks (only diagonal and tail tiles need them).
template <bool MASK>
__device__ __forceinline__ void dq_probs(const f32x4 (&s)[2], const f32x4 (&dp)[2], float c,
                                         float lse2, float Di, int key0, int g, int qrow, int Nk,
                                         int causal, int off, bf16x8& tf, bf16x8& rf) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float P = fexp2(fmaf(s[kb][i], c, -lse2));
            const __bf16 t = to_bf16(P * (dp[kb][i] - Di)), r = to_bf16(P);
            if constexpr (MASK) {
                // select, not multiply: a masked pair contributes exactly 0
                // whatever its logit, dP or LDS row held
                const int key = key0 + kb * 16 + 4 * g + i;
                const bool ok = key < Nk && (!causal || key <= qrow + off);
                tf[kb * 4 + i] = ok ? t : (__bf16)0.0f;
                rf[kb * 4 + i] = ok ? r : (__bf16)0.0f;
            } else {
                tf[kb * 4 + i] = t;
                rf[kb * 4 + i] = r;
            }
        }
}

template <int D, bool GPROJ, bool WRITE_Z, int NB = 2>
__global__ __launch_bounds__(kThreads * 2 / NB, D == 64 ? GPA_DQ_OCC64 : 2 / NB)
void bwd_dq_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ O,
    const uint16_t* __restrict__ dO, const float* __restrict__ LSE, float* __restrict__ D_out,
    float* __restrict__ TS, uint16_t* __restrict__ dQ,
    float* __restrict__ rho_out, float* __restrict__ m_out, float* __restrict__ lam_out,
    uint16_t* __restrict__ Zout, int BH, int Nmax, int causal, float scale, int G,
    const int* __restrict__ cu, int Hq, int total, const int* __restrict__ cu_k, int total_k,
    int Nkmax) {
    constexpr int MB = D / 16;  // 16-column blocks of d
    constexpr int KC = D / 32;  // 32-wide k chunks of d
    constexpr int PER_NB = 2 * MB * 4 + 2;  // partial A, B (interleaved) and rho, m
    // NB 16-row query blocks per wave: QG groups of waves own the 64 rows,
    // two waves (the two key halves of each tile) per group.
    constexpr int QG = 4 / NB;
    constexpr int NTHR = 64 * 2 * QG;
    // A three-slot ring of [K tile, V tile] (row-major, swizzled): while tile
    // i is computed on, tiles i+1 and i+2 are in flight.  Slot 0 is reused at
    // the end for the pairwise reduction.
    constexpr int TILE_E = kTile * D;
    __shared__ __attribute__((aligned(16))) uint16_t S0[2 * TILE_E];
    __shared__ __attribute__((aligned(16))) uint16_t S1[2 * TILE_E];
    __shared__ __attribute__((aligned(16))) uint16_t S2[2 * TILE_E];

    const int T = (Nmax + kTile - 1) / kTile;  // tiles of the longest problem
    int bh, tile;
    map_block(blockIdx.x, BH, T, causal != 0, &bh, &tile);
    const SeqRows sr = seq_rows(cu, cu_k, bh, Nmax, Nkmax, G, Hq, total, total_k);
    const int N = sr.nq, Nk = sr.nk;
    if (tile * kTile >= N) return;  // a shorter sequence has no such tile
    const int off = Nk - N;           // causal: query i sees key j iff j <= i + off
    const size_t hoff = sr.q0 * D;    // query head
    const size_t kvoff = sr.kv0 * D;  // its key/value head
    const size_t soff = sr.q0;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int qh = wave % QG;  // which 16 NB-row group of the workgroup's 64 queries
    const int kh = wave / QG;  // which 32 of each 64-key tile
    const int q0w = tile * kTile + 16 * NB * qh;

    // Q^T and dO^T as B operands: column = this lane's query of block nb, k = d.
    // Rows beyond N load as zero.
    const uint32_t tbytes = (uint32_t)N * (2 * D);
    const rsrc_t rq = make_rsrc(Q + hoff, tbytes);
    const rsrc_t ru = make_rsrc(dO + hoff, tbytes);
    const rsrc_t ro = make_rsrc(O + hoff, tbytes);
    bf16x8 qf[NB][KC], uf[NB][KC];
    float lse2[NB], Di[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int qrow = q0w + nb * 16 + c16;
        float dpart = 0.f;
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
            const u32x4 qw = ld_row16<D>(rq, qrow, kc * 32 + 8 * g);
            const u32x4 uw = ld_row16<D>(ru, qrow, kc * 32 + 8 * g);
            const u32x4 ow = ld_row16<D>(ro, qrow, kc * 32 + 8 * g);
            qf[nb][kc] = __builtin_bit_cast(bf16x8, qw);
            uf[nb][kc] = __builtin_bit_cast(bf16x8, uw);
            // Algorithm 1's preprocessing, fused: D_i = sum_c fl32(dO_ic O_ic);
            // BF16 x BF16 products are exact in FP32.
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                dpart += lo_bf16(uw[e]) * lo_bf16(ow[e]);
                dpart += hi_bf16(uw[e]) * hi_bf16(ow[e]);
            }
        }
        Di[nb] = xor_sum(dpart);
        // Rows beyond N get log2-LSE = +inf, so every P of theirs is exactly 0.
        lse2[nb] = qrow < N ? LSE[soff + qrow] * kLog2e : INFINITY;
    }
    const float c = scale * kLog2e;
    const bf16x8 ones = ones_row0(c16);

    f32x4 accA[NB][MB], accB[NB][GPROJ ? MB : 1], accR[NB], accM[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) accA[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int mb = 0; mb < (GPROJ ? MB : 1); ++mb) accB[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
        accR[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        accM[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Only the last one or two key tiles need masks (the causal diagonal, the
    // key tail).  Query rows beyond N need none (their P is 0 and they are not
    // stored), nor do queries that see no key (the forward gave them
    // LSE = +inf).
    const KeyRange kr = key_range(tile, Nk, off, causal);
    const int nkv = kr.nkv, nplain = kr.nplain;

    TileDma<D, NTHR> dma;
    dma.init(lane, wave);
    // Piece j of the fill of `slot` with key tile kt (K calls, then V calls);
    // past the last tile it is a zero fill, so every step issues FILL_VM loads.
    constexpr int CALLS = TileDma<D, NTHR>::CALLS;
    constexpr int FILL_VM = 2 * CALLS;
    auto fill_piece = [&](uint16_t* slot, int kt, int j) {
        if (j < FILL_VM) {
            const int t = j / CALLS, k = j % CALLS;
            dma.load_call(t ? V + kvoff : K + kvoff, slot + t * TILE_E, kt * kTile, Nk, kt < nkv, k);
        }
    };
    // The register operands above must have arrived before the first fill: the
    // compiler cannot count the fills, so it must have nothing left to wait
    // for inside the loop.
    wait_vm_lgkm0<0>();
#pragma unroll
    for (int j = 0; j < FILL_VM; ++j) fill_piece(S0, 0, j);
#pragma unroll
    for (int j = 0; j < FILL_VM; ++j) fill_piece(S1, 1, j);
    wait_vm_lgkm0<FILL_VM>();
    __builtin_amdgcn_s_barrier();
    // One key tile: compute on slot `cur` while the fill of tile kt + 2 into
    // `nxt2` is issued piece by piece; at the end tile kt + 1 has landed and
    // every wave is done with `cur`, which the next step refills.
    auto step = [&](auto masked, int kt, const uint16_t* cur, uint16_t* nxt2) {
        constexpr bool MASK = decltype(masked)::value;
        const int k0 = kt * kTile;
        const uint16_t* Kc = cur;
        const uint16_t* Vc = cur + TILE_E;
        fill_piece(nxt2, kt + 2, 0);
        // In the gproj modes the transposed K operands of the A/B products are
        // read now, so their LDS latency hides behind the S/dP products and the
        // exponentials (measured faster there, slower in plain mode).
        constexpr int PF = (GPROJ && D == 64) ? MB : 0;
        bf16x8 ktr[PF > 0 ? PF : 1];
#pragma unroll
        for (int mb = 0; mb < PF; ++mb) ktr[mb] = ld_tr_operand<D>(Kc, 32 * kh, mb * 16, c16, g);
        // S^T = K Q^T and dP^T = V dO^T for this wave's 32 keys x 32 queries:
        // s[nb][kb] holds keys 4g+i of key block kb for query block nb.
        // Raise this wave's issue priority while it feeds the matrix core, so
        // that the other wave on the SIMD fills the vector ALU meanwhile.
        __builtin_amdgcn_s_setprio(1);
        // d = 128: LLVM's MFMA/LDS interleaving strategy 1 (measured 4-5 %
        // faster there in every mode; neutral at d = 64, which keeps the
        // default schedule).
        if constexpr (D == 128) __builtin_amdgcn_iglp_opt(1);
        f32x4 s[NB][2], dp[NB][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                s[nb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
                dp[nb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const int row = 32 * kh + kb * 16 + c16;
                const bf16x8 ka = ld_b128(Kc + tile_off<D>(row, kc * 32 + 8 * g));
                const bf16x8 va = ld_b128(Vc + tile_off<D>(row, kc * 32 + 8 * g));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    s[nb][kb] = mfma_16x16x32(ka, qf[nb][kc], s[nb][kb]);
                    dp[nb][kb] = mfma_16x16x32(va, uf[nb][kc], dp[nb][kb]);
                }
            }
            fill_piece(nxt2, kt + 2, 1 + kb);
        }
        bf16x8 tf[NB], rf[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            dq_probs<MASK>(s[nb], dp[nb], c, lse2[nb], Di[nb], k0 + 32 * kh, g,
                           q0w + nb * 16 + c16, Nk, causal, off, tf[nb], rf[nb]);
        // A^T[d][query] += K^T[d][key] t^T[key][query] (and B^T with r); the
        // row sums rho, m come from a constant ones operand.
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const bf16x8 ka =
                mb < PF ? ktr[mb < PF ? mb : 0] : ld_tr_operand<D>(Kc, 32 * kh, mb * 16, c16, g);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                accA[nb][mb] = mfma_16x16x32(ka, tf[nb], accA[nb][mb]);
                if (GPROJ) accB[nb][mb] = mfma_16x16x32(ka, rf[nb], accB[nb][mb]);
            }
            fill_piece(nxt2, kt + 2, 3 + mb);
        }
        if (GPROJ) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                accR[nb] = mfma_16x16x32(ones, tf[nb], accR[nb]);
                accM[nb] = mfma_16x16x32(ones, rf[nb], accM[nb]);
            }
        }
        // Tile kt + 1 must have landed; tile kt + 2 may stay in flight.
        wait_vm_lgkm0<FILL_VM>();
        __builtin_amdgcn_s_barrier();
    };
    const std::false_type plain;
    const std::true_type masked;
    // Tile t lives in slot t mod 3; only the last one or two tiles need masks.
    int kt = 0;
    for (; kt < nplain; kt += 3) {
        step(plain, kt, S0, S2);
        if (kt + 1 < nplain) step(plain, kt + 1, S1, S0);
        if (kt + 2 < nplain) step(plain, kt + 2, S2, S1);
    }
    for (kt = nplain; kt < nkv; ++kt) {
        const int r = kt % 3;
        if (r == 0)
            step(masked, kt, S0, S2);
        else if (r == 1)
            step(masked, kt, S1, S0);
        else
            step(masked, kt, S2, S1);
    }
    // The zero fills issued by the last steps must land before slot 0 is
    // reused for the reduction.
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();

    // Add the partials of the two waves that own the same queries (one query
    // block at a time, to bound the LDS the exchange needs).
    float red[NB][PER_NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                red[nb][(mb * 4 + i) * 2] = accA[nb][mb][i];
                red[nb][(mb * 4 + i) * 2 + 1] = GPROJ ? accB[nb][mb][i] : 0.f;
            }
        red[nb][2 * MB * 4] = accR[nb][0];
        red[nb][2 * MB * 4 + 1] = accM[nb][0];
        if (nb) __syncthreads();  // the previous exchange has been read
        pair_reduce<PER_NB, sizeof(S0) / 4, QG>(red[nb], reinterpret_cast<float*>(S0), wave, lane);
    }
    if (wave >= QG) return;

#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int qrow = q0w + nb * 16 + c16;
        // rho and m of this lane's query sit in accumulator row 0 (lanes g == 0).
        float lam = 0.f, rho = 0.f, msum = 0.f;
        if (GPROJ) {
            rho = __shfl(red[nb][2 * MB * 4], c16);
            msum = __shfl(red[nb][2 * MB * 4 + 1], c16);
            lam = (msum != 0.f) ? rho / msum : 0.f;  // one IEEE FP32 division
        }
        if (qrow < N) {
            uint16_t* drow = dQ + hoff + (size_t)qrow * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                    const float a = red[nb][(mb * 4 + i) * 2];
                    const float b = red[nb][(mb * 4 + i) * 2 + 1];
                    if (GPROJ) {
                        const float corr = lam * b;
                        const float diff = a - corr;
                        v[i] = scale * diff;
                    } else {
                        v[i] = scale * a;
                    }
                }
                st_bf16x4(drow + mb * 16 + 4 * g, v[0], v[1], v[2], v[3]);
            }
            if (WRITE_Z) {
                // -z = BF16(fl32(-lambda q)) = -BF16(fl32(lambda q)) for the key
                // correction (negation is exact), so the key pass adds r^T (-z)
                // into the t^T Q accumulator: the lane holds d = kc*32 + 8g .. +7
                // of its query row.
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) {
                    bf16x8 z;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        z[e] = to_bf16(-lam * bf16_to_f32(qf[nb][kc][e]));
                    *reinterpret_cast<bf16x8*>(Zout + hoff + (size_t)qrow * D + kc * 32 + 8 * g) = z;
                }
            }
            if (g == 0) {
                D_out[soff + qrow] = Di[nb];
                rho_out[soff + qrow] = rho;
                m_out[soff + qrow] = msum;
                lam_out[soff + qrow] = lam;
            }
        }
        // The tile's statistics block for the key-major pass: log2-scaled LSE
        // (+inf beyond N), then D (0 beyond N).
        if (g == 0) {
            float* ts = TS + ((size_t)bh * T + tile) * kStatFloats;
            ts[qrow - tile * kTile] = lse2[nb];
            ts[kTile + qrow - tile * kTile] = Di[nb];
        }
    }
}

// ----------------------------------------------------------- key-major pass
// P, r, t of one 16-key x 16-query block: s, dp hold queries 4g+i of the
// block for this lane's key; they fill half `half` of the B operands tf, rf.
// Query rows beyond N, and queries that see no key, have log2-LSE = +inf
// (P = 0); key rows beyond the key count are never stored; so only the causal
// diagonal needs a mask: key krow is visible to query qrow iff
// krow <= qrow + off.
template <bool MASK>
__device__ __forceinline__ void dkdv_probs(const f32x4& s, const f32x4& dp, const f32x4& l2,
                                           const f32x4& dd, float c, int qb, int g, int krow,
                                           int off, int half, bf16x8& tf, bf16x8& rf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float P = fexp2(fmaf(s[i], c, -l2[i]));
        const __bf16 t = to_bf16(P * (dp[i] - dd[i])), r = to_bf16(P);
        if constexpr (MASK) {
            // select, not multiply: a masked pair contributes exactly 0
            const bool ok = krow <= qb + 4 * g + i + off;
            tf[half * 4 + i] = ok ? t : (__bf16)0.0f;
            rf[half * 4 + i] = ok ? r : (__bf16)0.0f;
        } else {
            tf[half * 4 + i] = t;
            rf[half * 4 + i] = r;
        }
    }
}

// FUSED_DQ (dense multi-head only): the single key-major pass of Algorithm 1's
// first loop.  Besides dV and dK it forms this key tile's share of A = tK for
// every query tile it visits and adds it into the FP32 accumulator dQacc
// [BH, N, d] with device-scope atomic adds (dQ is formed afterwards).  t goes
// through LDS once per step, as the transposed operand of that product.  With
// GPROJ as well it is that loop with the GProj additions: B = rK into Bacc
// (r through LDS like t) and the row masses rho = sum t, m = sum r into
// rho_acc, m_acc, all by atomic adds; the key correction is then a second
// pass (bwd_dk_corr_kernel), so the FP32 dK^acc = t^T Q goes to dKacc
// unscaled when dKacc is given (else dK = BF16(alpha dK^acc), as in plain).
template <int D, bool GPROJ, bool FUSED_DQ = false>
__global__ __launch_bounds__(kThreads, D == 64 ? GPA_DKDV_OCC64 : 1) void bwd_dkdv_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
    const float* __restrict__ TS, const uint16_t* __restrict__ Z, uint16_t* __restrict__ dK,
    uint16_t* __restrict__ dV, float* __restrict__ dKp, float* __restrict__ dVp, int BH, int Nmax,
    int causal, float scale, int G, const int* __restrict__ cu, int Hq, int total,
    const int* __restrict__ cu_k, int total_k, int Nkmax, float* __restrict__ dQacc = nullptr,
    float* __restrict__ Bacc = nullptr, float* __restrict__ rho_acc = nullptr,
    float* __restrict__ m_acc = nullptr, float* __restrict__ dKacc = nullptr) {
    constexpr int MB = D / 16;
    constexpr int KC = D / 32;
    // ZC: the two-pass schedule's key correction, folded into this pass (Z
    // staged, r^T (-z) added into the t^T Q accumulator).  AB: the atomic
    // schedule's B, rho and m.
    constexpr bool ZC = GPROJ && !FUSED_DQ;
    constexpr bool AB = GPROJ && FUSED_DQ;
    // d = 128 runs one wave per SIMD: order each step for the wave's own
    // overlap of vector and matrix work (see the step).
    constexpr bool PIPE = D == 128 && !FUSED_DQ;
    constexpr int NT = ZC ? 3 : 2;  // staged tensors: Q, dO (and Z = BF16(lambda Q))
    // Accumulators per output element: dV, and dK^acc - C in one (the GProj
    // pass adds t^T Q and r^T (-z) into the same FP32 accumulator).
    constexpr int NV = 2;
    constexpr int PER_KB = NV * MB * 4;
    // One ring slot: the NT query-tile tensors, then per wave the row
    // statistics of its 32 queries (32 log2-LSE, 32 D as FP32).  Three slots in
    // three separate LDS objects (so the compiler can tell the slot being read
    // from those the DMA is filling): while tile i is computed on, tiles i+1
    // and i+2 are in flight, which gives every load two steps to land.
    constexpr int TILE_E = kTile * D;  // BF16 elements of one staged tensor
    constexpr int STAT_E = kWaves * 128;  // 4 x 256 bytes of statistics
    constexpr int SLOT_E = NT * TILE_E + STAT_E;
    __shared__ __attribute__((aligned(16))) uint16_t B0[SLOT_E];
    __shared__ __attribute__((aligned(16))) uint16_t B1[SLOT_E];
    __shared__ __attribute__((aligned(16))) uint16_t B2[SLOT_E];
    // fused dQ: this tile's keys [key][d] and the step's t as [key][query]
    __shared__ __attribute__((aligned(16))) uint16_t Ks[FUSED_DQ ? TILE_E : 8];
    __shared__ __attribute__((aligned(16))) uint16_t Xt[FUSED_DQ ? kTile * kTile : 8];
    __shared__ __attribute__((aligned(16))) uint16_t Xr[AB ? kTile * kTile : 8];

    const int Tq = (Nmax + kTile - 1) / kTile;   // query tiles of the longest problem
    const int Tk = (Nkmax + kTile - 1) / kTile;  // key tiles of the longest problem
    int bh, tile;
    map_block(blockIdx.x, BH, Tk, false, &bh, &tile);
    const SeqRows sr = seq_rows(cu, cu_k, bh, Nmax, Nkmax, G, Hq, total, total_k);
    const int N = sr.nq, Nk = sr.nk;
    if (tile * kTile >= Nk) return;  // a shorter sequence has no such tile
    const int T = (N + kTile - 1) / kTile;
    const int off = Nk - N;           // causal: query i sees key j iff j <= i + off
    const size_t hoff = sr.q0 * D;    // query head: Q, dO, z
    const size_t kvoff = sr.kv0 * D;  // its key/value head: K, V, dK, dV
    const size_t poff = sr.p0 * D;    // this query head's partials over the key rows
    const float* tsh = TS + (size_t)bh * Tq * kStatFloats;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int kh = wave & 1;   // which 32 of the workgroup's 64 keys
    const int qh = wave >> 1;  // which 32 of each 64-query tile
    const int k0w = tile * kTile + 32 * kh;

    // K^T and V^T as B operands: column = this lane's key of block kb, k = d.
    // Rows beyond the key count load as zero.
    const uint32_t tbytes = (uint32_t)Nk * (2 * D);
    const rsrc_t rk = make_rsrc(K + kvoff, tbytes);
    const rsrc_t rv = make_rsrc(V + kvoff, tbytes);
    bf16x8 kf[2][KC], vf[2][KC];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
            const int krow = k0w + kb * 16 + c16;
            kf[kb][kc] = __builtin_bit_cast(bf16x8, ld_row16<D>(rk, krow, kc * 32 + 8 * g));
            vf[kb][kc] = __builtin_bit_cast(bf16x8, ld_row16<D>(rv, krow, kc * 32 + 8 * g));
        }
    const float c = scale * kLog2e;

    f32x4 accV[2][MB], accK[2][MB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            accV[kb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            accK[kb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }

    // The first query tile that sees a key of this tile.  The causal boundary
    // crosses at most the first two query tiles; without causal no query is
    // masked (a mask offset no row reaches).
    const int qt0 = causal ? max(0, floor_div(tile * kTile - off, kTile)) : 0;
    const int moff = causal ? off : (1 << 30);
    const uint16_t* src[NT];
    src[0] = Q + hoff;
    src[1] = dO + hoff;
    if (ZC) src[NT - 1] = Z + hoff;

    TileDma<D> dma;
    dma.init(lane, wave);
    // Vector-memory instructions one slot fill issues per wave: NT tensors of
    // TileDma::CALLS each, plus one for the statistics.  Every step issues one
    // fill (a zero fill past the last tile), so the count between a fill and
    // the wait for it is always FILL_VM.  Rows beyond N arrive as zeros.
    constexpr int FILL_VM = NT * TileDma<D>::CALLS + 1;
    // Piece j (0 <= j < FILL_VM) of a fill: the statistics first, then the
    // tensors' calls in order.  A step spreads its fill's pieces over its
    // compute so the loads do not all queue at once.
    auto fill_piece = [&](uint16_t* slot, int qt, int j) {
        const bool valid = qt < T;
        if (j == 0) {
            stat_dma(tsh + (size_t)(valid ? qt : 0) * kStatFloats,
                     reinterpret_cast<float*>(slot + NT * TILE_E) + 64 * wave, lane, qh, valid);
        } else if (j < FILL_VM) {
            const int t = (j - 1) / TileDma<D>::CALLS, k = (j - 1) % TileDma<D>::CALLS;
            dma.load_call(src[t], slot + t * TILE_E, qt * kTile, N, valid, k);
        }
    };
    auto fill = [&](uint16_t* slot, int qt) {
#pragma unroll
        for (int j = 0; j < FILL_VM; ++j) fill_piece(slot, qt, j);
    };
    // The register operands above must have arrived before the first fill: the
    // compiler cannot count the fills, so it must have nothing left to wait
    // for inside the loop.
    wait_vm_lgkm0<0>();
    if constexpr (FUSED_DQ) {
        dma.load(K + kvoff, Ks, tile * kTile, Nk);
        wait_vm_lgkm0<0>();
    }
    const rsrc_t rdq = make_rsrc(FUSED_DQ ? dQacc + hoff : nullptr,
                                 FUSED_DQ ? (uint32_t)N * (uint32_t)D * 4u : 0u);
    const rsrc_t rdb = make_rsrc(AB ? Bacc + hoff : nullptr, AB ? (uint32_t)N * (uint32_t)D * 4u : 0u);
    const rsrc_t rrho = make_rsrc(AB ? rho_acc + sr.q0 : nullptr, AB ? (uint32_t)N * 4u : 0u);
    const rsrc_t rms = make_rsrc(AB ? m_acc + sr.q0 : nullptr, AB ? (uint32_t)N * 4u : 0u);
    fill(B0, qt0);
    fill(B1, qt0 + 1);
    wait_vm_lgkm0<FILL_VM>();
    __builtin_amdgcn_s_barrier();

    // One query tile: compute on slot `cur` while slot `nxt2` receives tile
    // qt + 2; at the end, tile qt + 1 has landed and every wave is done with
    // `cur`, which the next step refills.
    auto step = [&](auto masked, int qt, const uint16_t* cur, uint16_t* nxt2) {
        constexpr bool MASK = decltype(masked)::value;
        const int q0 = qt * kTile;
        // The fill of tile qt + 2 is issued in pieces through the step (a few
        // first, one after each S/dP block, the rest in the dV/dK phase); it
        // has until the end of step qt + 1 to land.
        constexpr int AT_START = FILL_VM > 6 ? FILL_VM - 6 : 1;
#pragma unroll
        for (int j = 0; j < AT_START; ++j) fill_piece(nxt2, qt + 2, j);
        const uint16_t* Qc = cur;
        const uint16_t* Uc = cur + TILE_E;
        const uint16_t* Zc = cur + (NT - 1) * TILE_E;
        const float* st = reinterpret_cast<const float*>(cur + NT * TILE_E) + 64 * wave;
        f32x4 l2[2], dd[2];
#pragma unroll
        for (int mq = 0; mq < 2; ++mq) {
            l2[mq] = *reinterpret_cast<const f32x4*>(st + mq * 16 + 4 * g);
            dd[mq] = *reinterpret_cast<const f32x4*>(st + 32 + mq * 16 + 4 * g);
        }
        bf16x8 tf[2], rf[2];
        if constexpr (PIPE) {
            // One wave per SIMD (d = 128): no second wave fills the vector
            // ALU while this one multiplies, so the step is ordered by key
            // block instead, for the wave's own co-issue: S/dP of key block 0,
            // then S/dP of block 1 beside the probabilities of block 0, then
            // the dV/dK/C products of block 0 beside the probabilities of
            // block 1, then the products of block 1.  Every accumulator still
            // receives its products in the same order.
            bf16x8 qa[2][KC], ua[2][KC];
#pragma unroll
            for (int mq = 0; mq < 2; ++mq)
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) {
                    const int row = 32 * qh + mq * 16 + c16;
                    qa[mq][kc] = ld_b128(Qc + tile_off<D>(row, kc * 32 + 8 * g));
                    ua[mq][kc] = ld_b128(Uc + tile_off<D>(row, kc * 32 + 8 * g));
                }
            // LLVM's small-GEMM interleaving strategy for this order (measured
            // 3-4 % faster than strategy 1 here, which pairs each product with
            // an LDS read issued just before it).
            __builtin_amdgcn_iglp_opt(0);
            f32x4 sv[2][2], dpv[2][2];  // [kb][mq]
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int mq = 0; mq < 2; ++mq) {
                    sv[kb][mq] = f32x4{0.f, 0.f, 0.f, 0.f};
                    dpv[kb][mq] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kc = 0; kc < KC; ++kc) {
                        sv[kb][mq] = mfma_16x16x32(qa[mq][kc], kf[kb][kc], sv[kb][mq]);
                        dpv[kb][mq] = mfma_16x16x32(ua[mq][kc], vf[kb][kc], dpv[kb][mq]);
                    }
                    fill_piece(nxt2, qt + 2, AT_START + kb * 2 + mq);
                }
            }
            // The transposed A operands of every column block, held for both
            // key blocks.
            bf16x8 opd[MB][NT];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                opd[mb][0] = ld_tr_operand<D>(Uc, 32 * qh, mb * 16, c16, g);
                opd[mb][1] = ld_tr_operand<D>(Qc, 32 * qh, mb * 16, c16, g);
                if (ZC) opd[mb][NT - 1] = ld_tr_operand<D>(Zc, 32 * qh, mb * 16, c16, g);
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int mq = 0; mq < 2; ++mq)
                    dkdv_probs<MASK>(sv[kb][mq], dpv[kb][mq], l2[mq], dd[mq], c,
                                     q0 + 32 * qh + mq * 16, g, k0w + kb * 16 + c16, moff, mq,
                                     tf[kb], rf[kb]);
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    accV[kb][mb] = mfma_16x16x32(opd[mb][0], rf[kb], accV[kb][mb]);
                    accK[kb][mb] = mfma_16x16x32(opd[mb][1], tf[kb], accK[kb][mb]);
                    if (ZC) accK[kb][mb] = mfma_16x16x32(opd[mb][NT - 1], rf[kb], accK[kb][mb]);
                    if (kb == 1) fill_piece(nxt2, qt + 2, AT_START + 4 + mb);
                }
            }
        } else {
            // The transposed A operands of the first two column blocks of the
            // dV/dK/C products are read now, so their LDS latency hides behind the
            // S/dP products and the exponentials.
            bf16x8 opd[2][NT];
            auto read_ops = [&](bf16x8 (&o)[NT], int mb) {
                o[0] = ld_tr_operand<D>(Uc, 32 * qh, mb * 16, c16, g);
                o[1] = ld_tr_operand<D>(Qc, 32 * qh, mb * 16, c16, g);
                if (ZC) o[NT - 1] = ld_tr_operand<D>(Zc, 32 * qh, mb * 16, c16, g);
            };
            read_ops(opd[0], 0);
            read_ops(opd[1], 1);
            __builtin_amdgcn_sched_barrier(0);

            // S = Q K^T and dP = dO V^T for this wave's 32 queries x 32 keys, one
            // 16 x 16 block at a time: s holds queries 4g+i of query block mq for
            // key block kb, and P, r, t of that block go straight into half mq of
            // the key block's B operands tf[kb], rf[kb].
            // Raise this wave's issue priority while it feeds the matrix core, so
            // that the other wave on the SIMD fills the vector ALU meanwhile.
            __builtin_amdgcn_s_setprio(1);
            // LLVM's interleaving strategy 1 for matrix-core and LDS instructions
            // (measured 1.5-2 % faster here; neutral in the query pass).
            __builtin_amdgcn_iglp_opt(1);
    #pragma unroll
            for (int mq = 0; mq < 2; ++mq) {
                const int row = 32 * qh + mq * 16 + c16;
                bf16x8 qa[KC], ua[KC];
    #pragma unroll
                for (int kc = 0; kc < KC; ++kc) {
                    qa[kc] = ld_b128(Qc + tile_off<D>(row, kc * 32 + 8 * g));
                    ua[kc] = ld_b128(Uc + tile_off<D>(row, kc * 32 + 8 * g));
                }
    #pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    f32x4 sv = {0.f, 0.f, 0.f, 0.f}, dpv = {0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                    for (int kc = 0; kc < KC; ++kc) {
                        sv = mfma_16x16x32(qa[kc], kf[kb][kc], sv);
                        dpv = mfma_16x16x32(ua[kc], vf[kb][kc], dpv);
                    }
                    dkdv_probs<MASK>(sv, dpv, l2[mq], dd[mq], c, q0 + 32 * qh + mq * 16, g,
                                     k0w + kb * 16 + c16, moff, mq, tf[kb], rf[kb]);
                    fill_piece(nxt2, qt + 2, AT_START + mq * 2 + kb);
                }
            }
            // dV^T[dv][key] += dO^T r ; dK^T += Q^T t ; C^T += Z^T r.  The A operands
            // of column block mb + 2 are read from LDS while block mb multiplies.
            __builtin_amdgcn_s_setprio(0);
    #pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const bf16x8* o = opd[mb & 1];
                const bf16x8 ua = o[0], qa = o[1], za = o[NT - 1];
    #pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    accV[kb][mb] = mfma_16x16x32(ua, rf[kb], accV[kb][mb]);
                    accK[kb][mb] = mfma_16x16x32(qa, tf[kb], accK[kb][mb]);
                    if (ZC) accK[kb][mb] = mfma_16x16x32(za, rf[kb], accK[kb][mb]);
                }
                if (mb + 2 < MB) read_ops(opd[mb & 1], mb + 2);
                fill_piece(nxt2, qt + 2, AT_START + 4 + mb);
            }
        }
        if constexpr (FUSED_DQ) {
            // t of this wave's 32 keys x 32 queries into Xt[key][query] (r
            // into Xr): lane (c16, g) holds key 32 kh + 16 kb + c16 at queries
            // 32 qh + 16 mq + 4 g + i, i.e. 8 contiguous bytes of one Xt row
            // per (kb, mq).  Keys beyond the key count (the tail of the last
            // key tile, which without causal masking no step masks) get
            // t = r = 0 here: their K rows load as zero, but their P would
            // still enter the row masses rho and m.
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int mq = 0; mq < 2; ++mq) {
                    const uint64_t keep = k0w + 16 * kb + c16 < Nk ? ~0ull : 0ull;
                    bf16x4 w4, r4;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        w4[i] = tf[kb][4 * mq + i];
                        r4[i] = rf[kb][4 * mq + i];
                    }
                    const int xo = tile_off<kTile>(32 * kh + 16 * kb + c16, 32 * qh + 16 * mq + 4 * g);
                    *reinterpret_cast<uint64_t*>(Xt + xo) = __builtin_bit_cast(uint64_t, w4) & keep;
                    if (AB)
                        *reinterpret_cast<uint64_t*>(Xr + xo) = __builtin_bit_cast(uint64_t, r4) & keep;
                }
            __syncthreads();
            // A block of this tile's share of A = tK (and B = rK): wave w takes
            // queries 16 w .. 16 w + 15 against all 64 keys.  Operands:
            // t[query][key] and K[key][d], both read transposed (key along k).
            // rho and m: the same t, r operands against a B operand whose
            // column 0 is ones, so accumulator column 0 holds the row sums.
            f32x4 aq[MB], bq[AB ? MB : 1], rsum = {0.f, 0.f, 0.f, 0.f}, msum = rsum;
#pragma unroll
            for (int db = 0; db < MB; ++db) aq[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int db = 0; db < (AB ? MB : 1); ++db) bq[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const bf16x8 ta = ld_tr_operand<kTile>(Xt, 32 * kc, 16 * wave, c16, g);
                bf16x8 ra = ta;
                if (AB) ra = ld_tr_operand<kTile>(Xr, 32 * kc, 16 * wave, c16, g);
#pragma unroll
                for (int db = 0; db < MB; ++db) {
                    const bf16x8 kop = ld_tr_operand<D>(Ks, 32 * kc, 16 * db, c16, g);
                    aq[db] = mfma_16x16x32(ta, kop, aq[db]);
                    if (AB) bq[db] = mfma_16x16x32(ra, kop, bq[db]);
                }
                if (AB) {
                    const bf16x8 ones = ones_row0(c16);
                    rsum = mfma_16x16x32(ta, ones, rsum);
                    msum = mfma_16x16x32(ra, ones, msum);
                }
            }
            // FP32 atomic adds through a buffer resource over this head's N
            // rows (rows beyond N are dropped by the range check): lanes c16
            // cover 16 consecutive columns of one query row, 64 contiguous
            // bytes per row and instruction.
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int qr = q0 + 16 * wave + 4 * g + i;
                const uint32_t off = (uint32_t)(qr * D + c16) * 4u;
#pragma unroll
                for (int db = 0; db < MB; ++db) {
                    __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(aq[db][i], rdq, off + 64u * db, 0,
                                                                    0);
                    if (AB)
                        __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(bq[db][i], rdb,
                                                                        off + 64u * db, 0, 0);
                }
                // the row sums sit in accumulator column 0 (lanes c16 == 0)
                if (AB && c16 == 0) {
                    __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(rsum[i], rrho, (uint32_t)qr * 4u, 0,
                                                                    0);
                    __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(msum[i], rms, (uint32_t)qr * 4u, 0,
                                                                    0);
                }
            }
            // The atomics share the vector-memory counter with the tile
            // fills; wait for everything rather than rely on the order in
            // which writes and loads complete.
            wait_vm_lgkm0<0>();
        } else {
            // Tile qt + 1 must have landed; tile qt + 2 may stay in flight.
            wait_vm_lgkm0<FILL_VM>();
        }
        __builtin_amdgcn_s_barrier();
    };
    const std::false_type plain;
    const std::true_type masked;
    // Tile t lives in slot (t - qt0) mod 3; the first two steps take the mask.
    // A key tile that no query sees (qt0 >= T) takes no step and stores zeros.
    if (qt0 < T) step(masked, qt0, B0, B2);
    if (qt0 + 1 < T) step(masked, qt0 + 1, B1, B0);
    for (int qt = qt0 + 2; qt < T; qt += 3) {
        step(plain, qt, B2, B1);
        if (qt + 1 < T) step(plain, qt + 1, B0, B2);
        if (qt + 2 < T) step(plain, qt + 2, B1, B0);
    }
    // The zero fills issued by the last steps must land before B0 is reused
    // for the reduction.
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();

    // Add the partials of the two waves that own the same keys (one key block
    // at a time, to bound the LDS the exchange needs).
    float red[2][PER_KB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = (mb * 4 + i) * NV;
                red[kb][j] = accV[kb][mb][i];
                red[kb][j + 1] = accK[kb][mb][i];
            }
        if (kb) __syncthreads();  // the previous exchange has been read
        pair_reduce<PER_KB, sizeof(B0) / 4>(red[kb], reinterpret_cast<float*>(B0), wave, lane);
    }
    if (wave >= 2) return;

#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int krow = k0w + kb * 16 + c16;
        if (krow >= Nk) continue;
        if (G > 1) {
            // This query head's FP32 contributions; the group sum casts them.
            float* vp = dVp + poff + (size_t)krow * D;
            float* kp = dKp + poff + (size_t)krow * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                f32x4 dv, dk;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                    const int j = (mb * 4 + i) * NV;
                    dv[i] = red[kb][j];
                    dk[i] = red[kb][j + 1];
                }
                *reinterpret_cast<f32x4*>(vp + mb * 16 + 4 * g) = dv;
                *reinterpret_cast<f32x4*>(kp + mb * 16 + 4 * g) = dk;
            }
            continue;
        }
        if (AB && dKacc != nullptr) {
            // the FP32 dK^acc for the correction pass, unscaled; dV final
            float* kp = dKacc + kvoff + (size_t)krow * D;
            uint16_t* vrow = dV + kvoff + (size_t)krow * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                f32x4 dk;
                float dv[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = (mb * 4 + i) * NV;
                    dv[i] = red[kb][j];
                    dk[i] = red[kb][j + 1];
                }
                *reinterpret_cast<f32x4*>(kp + mb * 16 + 4 * g) = dk;
                st_bf16x4(vrow + mb * 16 + 4 * g, dv[0], dv[1], dv[2], dv[3]);
            }
            continue;
        }
        uint16_t* vrow = dV + kvoff + (size_t)krow * D;
        uint16_t* krw = dK + kvoff + (size_t)krow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            float dv[4], dk[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                const int j = (mb * 4 + i) * NV;
                dv[i] = red[kb][j];
                dk[i] = scale * red[kb][j + 1];
            }
            st_bf16x4(vrow + mb * 16 + 4 * g, dv[0], dv[1], dv[2], dv[3]);
            st_bf16x4(krw + mb * 16 + 4 * g, dk[0], dk[1], dk[2], dk[3]);
        }
    }
}

// Second key-major pass of the atomic GProj schedule (Algorithm 1's loop for
// the key correction; eq. gproj-key-implemented), dense multi-head.  With
// lambda known, it rebuilds P and r-tilde for every causal pair with the first
// pass's instructions (so r-tilde = r bitwise), accumulates -C = r^T (-z) in
// FP32 over the query tiles and writes
// dK = BF16(fl32[alpha fl32(dK^acc - C)]) from the first pass's FP32 dK^acc.
// Same work split, ring and statistics staging as bwd_dkdv_kernel, with two
// staged tensors (Q for the logits, -z for the product) and no dP.
template <int D>
__global__ __launch_bounds__(kThreads, D == 64 ? 2 : 1) void bwd_dk_corr_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const float* __restrict__ TS, const uint16_t* __restrict__ Z,
    const float* __restrict__ dKacc, uint16_t* __restrict__ dK, int BH, int N, int causal,
    float scale) {
    constexpr int MB = D / 16;
    constexpr int KC = D / 32;
    constexpr int NT = 2;
    constexpr int TILE_E = kTile * D;
    constexpr int STAT_E = kWaves * 128;
    constexpr int SLOT_E = NT * TILE_E + STAT_E;
    __shared__ __attribute__((aligned(16))) uint16_t B0[SLOT_E];
    __shared__ __attribute__((aligned(16))) uint16_t B1[SLOT_E];
    __shared__ __attribute__((aligned(16))) uint16_t B2[SLOT_E];

    const int T = (N + kTile - 1) / kTile;
    int bh, tile;
    map_block(blockIdx.x, BH, T, false, &bh, &tile);
    const size_t hoff = (size_t)bh * N * D;
    const float* tsh = TS + (size_t)bh * T * kStatFloats;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int kh = wave & 1;
    const int qh = wave >> 1;
    const int k0w = tile * kTile + 32 * kh;

    const rsrc_t rk = make_rsrc(K + hoff, (uint32_t)N * (2 * D));
    bf16x8 kf[2][KC];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
            kf[kb][kc] = __builtin_bit_cast(
                bf16x8, ld_row16<D>(rk, k0w + kb * 16 + c16, kc * 32 + 8 * g));
    const float c = scale * kLog2e;
    f32x4 accC[2][MB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) accC[kb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // dense rows: a query tile below this key tile sees none of its keys
    const int qt0 = causal ? tile : 0;
    const int moff = causal ? 0 : (1 << 30);
    const uint16_t* src[NT] = {Q + hoff, Z + hoff};
    TileDma<D> dma;
    dma.init(lane, wave);
    constexpr int FILL_VM = NT * TileDma<D>::CALLS + 1;
    auto fill = [&](uint16_t* slot, int qt) {
        const bool valid = qt < T;
        stat_dma(tsh + (size_t)(valid ? qt : 0) * kStatFloats,
                 reinterpret_cast<float*>(slot + NT * TILE_E) + 64 * wave, lane, qh, valid);
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int k = 0; k < TileDma<D>::CALLS; ++k)
                dma.load_call(src[t], slot + t * TILE_E, qt * kTile, N, valid, k);
    };
    wait_vm_lgkm0<0>();
    fill(B0, qt0);
    fill(B1, qt0 + 1);
    wait_vm_lgkm0<FILL_VM>();
    __builtin_amdgcn_s_barrier();

    auto step = [&](auto masked, int qt, const uint16_t* cur, uint16_t* nxt2) {
        constexpr bool MASK = decltype(masked)::value;
        const int q0 = qt * kTile;
        fill(nxt2, qt + 2);
        const uint16_t* Qc = cur;
        const uint16_t* Zc = cur + TILE_E;
        const float* st = reinterpret_cast<const float*>(cur + NT * TILE_E) + 64 * wave;
        f32x4 l2[2];
#pragma unroll
        for (int mq = 0; mq < 2; ++mq) l2[mq] = *reinterpret_cast<const f32x4*>(st + mq * 16 + 4 * g);
        const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
        bf16x8 tf[2], rf[2];
#pragma unroll
        for (int mq = 0; mq < 2; ++mq) {
            const int row = 32 * qh + mq * 16 + c16;
            bf16x8 qa[KC];
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) qa[kc] = ld_b128(Qc + tile_off<D>(row, kc * 32 + 8 * g));
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                f32x4 sv = zero4;
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) sv = mfma_16x16x32(qa[kc], kf[kb][kc], sv);
                // the first pass's probability code; t is not used here
                dkdv_probs<MASK>(sv, zero4, l2[mq], zero4, c, q0 + 32 * qh + mq * 16, g,
                                 k0w + kb * 16 + c16, moff, mq, tf[kb], rf[kb]);
            }
        }
        // -C^T[d][key] += (-z)^T r
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const bf16x8 za = ld_tr_operand<D>(Zc, 32 * qh, mb * 16, c16, g);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) accC[kb][mb] = mfma_16x16x32(za, rf[kb], accC[kb][mb]);
        }
        wait_vm_lgkm0<FILL_VM>();
        __builtin_amdgcn_s_barrier();
    };
    const std::false_type plain;
    const std::true_type masked;
    if (qt0 < T) step(masked, qt0, B0, B2);
    if (qt0 + 1 < T) step(masked, qt0 + 1, B1, B0);
    for (int qt = qt0 + 2; qt < T; qt += 3) {
        step(plain, qt, B2, B1);
        if (qt + 1 < T) step(plain, qt + 1, B0, B2);
        if (qt + 2 < T) step(plain, qt + 2, B1, B0);
    }
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();

    constexpr int PER_KB = MB * 4;
    float red[2][PER_KB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[kb][mb * 4 + i] = accC[kb][mb][i];
        if (kb) __syncthreads();
        pair_reduce<PER_KB, sizeof(B0) / 4>(red[kb], reinterpret_cast<float*>(B0), wave, lane);
    }
    if (wave >= 2) return;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int krow = k0w + kb * 16 + c16;
        if (krow >= N) continue;
        const float* ka = dKacc + hoff + (size_t)krow * D;
        uint16_t* krw = dK + hoff + (size_t)krow * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(ka + mb * 16 + 4 * g);
            float dk[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
                const float diff = a[i] + red[kb][mb * 4 + i];  // dK^acc - C (-C accumulated)
                dk[i] = scale * diff;
            }
            st_bf16x4(krw + mb * 16 + 4 * g, dk[0], dk[1], dk[2], dk[3]);
        }
    }
}

// Group sum of the per-query-head FP32 contributions (G > 1): thread t of the
// grid owns 8 consecutive elements of one key/value head and adds the G query
// heads' values in head order, starting from zero; dK takes the scale after
// the sum, matching BF16(fl32[alpha (dK^acc - C)]) with dK^acc and C summed
// over the group.  A memory-bound pass: with the group size known at compile
// time (GC > 0) every load of the thread is issued before the first add.
template <int GC>
__global__ __launch_bounds__(256) void group_sum_kernel(const float* __restrict__ dKp,
                                                        const float* __restrict__ dVp,
                                                        uint16_t* __restrict__ dK,
                                                        uint16_t* __restrict__ dV, int BHkv,
                                                        int Grt, size_t per_head, float scale) {
    const int G = GC > 0 ? GC : Grt;
    const size_t octs = per_head / 8;
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (size_t)BHkv * octs) return;
    const size_t kvh = t / octs, e = (t - kvh * octs) * 8;
    const float* kp = dKp + kvh * G * per_head + e;
    const float* vp = dVp + kvh * G * per_head + e;
    f32x4 sk[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    f32x4 sv[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    if constexpr (GC > 0) {
        f32x4 lk[GC][2], lv[GC][2];
#pragma unroll
        for (int gq = 0; gq < GC; ++gq)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                lk[gq][h] = *reinterpret_cast<const f32x4*>(kp + gq * per_head + 4 * h);
                lv[gq][h] = *reinterpret_cast<const f32x4*>(vp + gq * per_head + 4 * h);
            }
#pragma unroll
        for (int gq = 0; gq < GC; ++gq)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                sk[h] += lk[gq][h];
                sv[h] += lv[gq][h];
            }
    } else {
        for (int gq = 0; gq < G; ++gq)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                sk[h] += *reinterpret_cast<const f32x4*>(kp + gq * per_head + 4 * h);
                sv[h] += *reinterpret_cast<const f32x4*>(vp + gq * per_head + 4 * h);
            }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        float k4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
            k4[i] = scale * sk[h][i];
        }
        st_bf16x4(dK + kvh * per_head + e + 4 * h, k4[0], k4[1], k4[2], k4[3]);
        st_bf16x4(dV + kvh * per_head + e + 4 * h, sv[h][0], sv[h][1], sv[h][2], sv[h][3]);
    }
}

// Preprocessing of the atomic schedule (dense multi-head): Algorithm 1's
// D_i = sum_c fl32(dO_ic O_ic) with the query-major pass's own lanes and
// summation order (so its bits, and hence t, equal that pass's), the per-tile
// statistics block the key-major pass stages, and zeroed accumulators: A
// (dQacc) always, B, rho and m when given (the GProj modes).
// One workgroup per (head, 64-row tile); wave w takes rows 16 w .. 16 w + 15.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_pre_kernel(const uint16_t* __restrict__ O,
                                                           const uint16_t* __restrict__ dO,
                                                           const float* __restrict__ LSE,
                                                           float* __restrict__ TS,
                                                           float* __restrict__ dQacc,
                                                           float* __restrict__ Bacc,
                                                           float* __restrict__ rho_acc,
                                                           float* __restrict__ m_acc, int BH,
                                                           int N) {
    constexpr int KC = D / 32;
    const int T = (N + kTile - 1) / kTile;
    const int bh = blockIdx.x / T, tile = blockIdx.x - bh * T;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int qrow = tile * kTile + 16 * wave + c16;
    const size_t hoff = (size_t)bh * N * D;
    const uint32_t tb = (uint32_t)N * (2 * D);
    const rsrc_t ru = make_rsrc(dO + hoff, tb);
    const rsrc_t ro = make_rsrc(O + hoff, tb);
    float dpart = 0.f;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
        const u32x4 uw = ld_row16<D>(ru, qrow, kc * 32 + 8 * g);
        const u32x4 ow = ld_row16<D>(ro, qrow, kc * 32 + 8 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            dpart += lo_bf16(uw[e]) * lo_bf16(ow[e]);
            dpart += hi_bf16(uw[e]) * hi_bf16(ow[e]);
        }
    }
    const float Di = xor_sum(dpart);
    if (g == 0) {
        float* ts = TS + ((size_t)bh * T + tile) * kStatFloats;
        ts[16 * wave + c16] = qrow < N ? LSE[(size_t)bh * N + qrow] * kLog2e : INFINITY;
        ts[kTile + 16 * wave + c16] = Di;
    }
    if (qrow < N) {
        float* a = dQacc + hoff + (size_t)qrow * D;
#pragma unroll
        for (int c = 0; c < D / 4; c += 4)
            *reinterpret_cast<f32x4*>(a + 4 * (c + g)) = f32x4{0.f, 0.f, 0.f, 0.f};
        if (Bacc != nullptr) {
            float* b = Bacc + hoff + (size_t)qrow * D;
#pragma unroll
            for (int c = 0; c < D / 4; c += 4)
                *reinterpret_cast<f32x4*>(b + 4 * (c + g)) = f32x4{0.f, 0.f, 0.f, 0.f};
            if (g == 0) {
                rho_acc[(size_t)bh * N + qrow] = 0.f;
                m_acc[(size_t)bh * N + qrow] = 0.f;
            }
        }
    }
}

// The atomic schedule's lambda and dQ (eq. gproj-query-implemented): per row
// lambda = rho / m (one IEEE FP32 division, 0 where m = 0) and
// dQ = BF16(fl32[alpha fl32(A - fl32(lambda B))]) from the FP32 accumulators;
// with Zneg also -z = BF16(fl32(-lambda q)) for the correction pass, and with
// lam_out lambda itself.  Thread t takes 8 consecutive elements of one row.
template <int D>
__global__ __launch_bounds__(256) void bwd_gproj_finalize_kernel(
    const float* __restrict__ A, const float* __restrict__ Bm, const float* __restrict__ rho,
    const float* __restrict__ msum, const uint16_t* __restrict__ Q, uint16_t* __restrict__ dQ,
    uint16_t* __restrict__ Zneg, float* __restrict__ lam_out, size_t rows, float scale) {
    constexpr int PER = D / 8;
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= rows * PER) return;
    const size_t row = t / PER;
    const int part = (int)(t - row * PER);
    const size_t e = row * D + 8 * part;
    const float m = msum[row];
    const float lam = (m != 0.f) ? rho[row] / m : 0.f;  // one IEEE FP32 division
    float v[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(A + e + 4 * h);
        const f32x4 b = *reinterpret_cast<const f32x4*>(Bm + e + 4 * h);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
            const float corr = lam * b[i];
            const float diff = a[i] - corr;
            v[4 * h + i] = scale * diff;
        }
    }
    st_bf16x4(dQ + e, v[0], v[1], v[2], v[3]);
    st_bf16x4(dQ + e + 4, v[4], v[5], v[6], v[7]);
    if (Zneg != nullptr) {
        const bf16x8 q = *reinterpret_cast<const bf16x8*>(Q + e);
        bf16x8 z;
#pragma unroll
        for (int i = 0; i < 8; ++i) z[i] = to_bf16(-lam * bf16_to_f32(q[i]));
        *reinterpret_cast<bf16x8*>(Zneg + e) = z;
    }
    if (lam_out != nullptr && part == 0) lam_out[row] = lam;
}

// dQ = BF16(fl32(alpha A)) from the FP32 accumulator, 4 elements per thread.
__global__ __launch_bounds__(256) void bwd_dq_finalize_kernel(const float* __restrict__ dQacc,
                                                              uint16_t* __restrict__ dQ,
                                                              size_t quads, float scale) {
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= quads) return;
    const f32x4 a = *reinterpret_cast<const f32x4*>(dQacc + 4 * t);
    float v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
        v[i] = scale * a[i];
    }
    st_bf16x4(dQ + 4 * t, v[0], v[1], v[2], v[3]);
}

}  // namespace

hipError_t launch_bwd_pre(const uint16_t* O, const uint16_t* dO, const float* LSE, float* TS,
                          const AtomicAcc& a, const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
    if (s.d == 64)
        launch_kernel(bwd_pre_kernel<64>, grid, block, st, O, dO, LSE, TS, a.A, a.B, a.rho, a.m,
                      s.BH, s.N);
    else
        launch_kernel(bwd_pre_kernel<128>, grid, block, st, O, dO, LSE, TS, a.A, a.B, a.rho, a.m,
                      s.BH, s.N);
    return hipGetLastError();
}

hipError_t launch_bwd_fused(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            const uint16_t* dO, const float* TS, uint16_t* dK, uint16_t* dV,
                            const AtomicAcc& a, int mode, const Shape& s, hipStream_t st) {
    const int Tk = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * Tk)), block(kThreads);
    float* dKacc = mode == 2 ? a.dKacc : nullptr;
#define GPA_FUSED(DD, GP)                                                                    \
    launch_kernel(bwd_dkdv_kernel<DD, GP, true>, grid, block, st, Q, K, V, dO, TS, nullptr,  \
                  dK, dV, nullptr, nullptr, s.BH, s.N, s.causal, s.scale, 1, nullptr, s.BH, 0, \
                  nullptr, 0, s.N, a.A, a.B, a.rho, a.m, dKacc)
    if (s.d == 64) {
        if (mode == 0) GPA_FUSED(64, false); else GPA_FUSED(64, true);
    } else {
        if (mode == 0) GPA_FUSED(128, false); else GPA_FUSED(128, true);
    }
#undef GPA_FUSED
    return hipGetLastError();
}

hipError_t launch_bwd_gproj_finalize(const AtomicAcc& a, const uint16_t* Q, uint16_t* dQ,
                                     uint16_t* Zneg, float* lam, const Shape& s, hipStream_t st) {
    const size_t rows = (size_t)s.BH * s.N;
    const size_t threads = rows * (size_t)(s.d / 8);
    dim3 grid((unsigned)((threads + 255) / 256)), block(256);
    if (s.d == 64)
        launch_kernel(bwd_gproj_finalize_kernel<64>, grid, block, st, a.A, a.B, a.rho, a.m, Q,
                      dQ, Zneg, lam, rows, s.scale);
    else
        launch_kernel(bwd_gproj_finalize_kernel<128>, grid, block, st, a.A, a.B, a.rho, a.m, Q,
                      dQ, Zneg, lam, rows, s.scale);
    return hipGetLastError();
}

hipError_t launch_bwd_dk_corr(const uint16_t* Q, const uint16_t* K, const float* TS,
                              const uint16_t* Zneg, const float* dKacc, uint16_t* dK,
                              const Shape& s, hipStream_t st) {
    const int Tk = (s.N + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * Tk)), block(kThreads);
    if (s.d == 64)
        launch_kernel(bwd_dk_corr_kernel<64>, grid, block, st, Q, K, TS, Zneg, dKacc, dK, s.BH,
                      s.N, s.causal, s.scale);
    else
        launch_kernel(bwd_dk_corr_kernel<128>, grid, block, st, Q, K, TS, Zneg, dKacc, dK, s.BH,
                      s.N, s.causal, s.scale);
    return hipGetLastError();
}

hipError_t launch_bwd_dq_finalize(const float* dQacc, uint16_t* dQ, const Shape& s,
                                  hipStream_t st) {
    const size_t quads = (size_t)s.BH * s.N * s.d / 4;
    dim3 grid((unsigned)((quads + 255) / 256)), block(256);
    launch_kernel(bwd_dq_finalize_kernel, grid, block, st, dQacc, dQ, quads, s.scale);
    return hipGetLastError();
}

hipError_t launch_bwd_dq(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* O, const uint16_t* dO, const float* LSE, float* Drow,
                         float* TS, uint16_t* dQ, float* rho, float* msum, float* lambda,
                         uint16_t* Z, int mode, const Shape& s, hipStream_t st) {
    const int T = (s.N + kTile - 1) / kTile;
    const int Nk = s.Nk > 0 ? s.Nk : s.N;
    dim3 grid((unsigned)(s.BH * T)), block(kThreads);
#define GPA_DQ(DD, GP, WZ, NB)                                                                \
    launch_kernel(bwd_dq_kernel<DD, GP, WZ, NB>, grid, block, st, Q, K, V, O, dO, LSE, Drow, TS, \
                  dQ, rho, msum, lambda, Z, s.BH, s.N, s.causal, s.scale, s.G, s.cu, s.Hq,    \
                  s.total, s.cu_k, s.total_k, Nk)
    if (s.d == 64) {
        if (mode == 2) GPA_DQ(64, true, true, 2);
        else if (mode == 1) GPA_DQ(64, true, false, 2);
        else GPA_DQ(64, false, false, 2);
    } else {
        // eight waves of one 16-row query block each (measured 5-8 % faster in
        // the GProj modes, bitwise the same outputs)
        block = dim3(2 * kThreads);
        if (mode == 2) GPA_DQ(128, true, true, 1);
        else if (mode == 1) GPA_DQ(128, true, false, 1);
        else GPA_DQ(128, false, false, 1);
    }
#undef GPA_DQ
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* dO, const float* TS, const uint16_t* Z,
                           uint16_t* dK, uint16_t* dV, float* dKp, float* dVp, int mode,
                           const Shape& s, hipStream_t st) {
    const int Nk = s.Nk > 0 ? s.Nk : s.N;
    const int Tk = (Nk + kTile - 1) / kTile;
    dim3 grid((unsigned)(s.BH * Tk)), block(kThreads);
    const bool gp = mode == 2;
#define GPA_DKDV(DD, GP)                                                                      \
    launch_kernel(bwd_dkdv_kernel<DD, GP>, grid, block, st, Q, K, V, dO, TS, Z, dK, dV, dKp, \
                  dVp, s.BH, s.N, s.causal, s.scale, s.G, s.cu, s.Hq, s.total, s.cu_k,       \
                  s.total_k, Nk, nullptr, nullptr, nullptr, nullptr, nullptr)
    if (s.d == 64) {
        if (gp) GPA_DKDV(64, true); else GPA_DKDV(64, false);
    } else {
        if (gp) GPA_DKDV(128, true); else GPA_DKDV(128, false);
    }
#undef GPA_DKDV
    return hipGetLastError();
}

hipError_t launch_bwd_group_sum(const float* dKp, const float* dVp, uint16_t* dK, uint16_t* dV,
                                const Shape& s, hipStream_t st) {
    const int BHkv = s.BH / s.G;
    const size_t per_head = (size_t)s.N * s.d;
    const size_t threads = (size_t)BHkv * (per_head / 8);
    dim3 grid((unsigned)((threads + 255) / 256)), block(256);
#define GPA_GSUM(GC)                                                                       \
    launch_kernel(group_sum_kernel<GC>, grid, block, st, dKp, dVp, dK, dV, BHkv, s.G, per_head, \
                  s.scale)
    if (s.G == 2) GPA_GSUM(2);
    else if (s.G == 4) GPA_GSUM(4);
    else if (s.G == 8) GPA_GSUM(8);
    else GPA_GSUM(0);
#undef GPA_GSUM
    return hipGetLastError();
}

}  // namespace gpa
