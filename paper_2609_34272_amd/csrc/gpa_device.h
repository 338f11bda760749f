// Device-side helpers shared by the gfx950 kernels of libgpa.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gpa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// FP32 log2(e), rounded to FP32.
constexpr float kLog2e = 1.44269504088896340736f;

// Tile geometry shared by the MFMA kernels.  A wave owns 16 or 32 rows of its
// operand (queries in the forward and the query-major backward, keys in the
// key-major backward); a workgroup has 4 waves (the d = 128 query-major pass,
// 8).
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kTile = 64;  // rows per workgroup tile and per streamed tile

__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 ld_b128(const uint16_t* p) {
    return *reinterpret_cast<const bf16x8*>(p);
}

// Two 8-byte reads joined into one MFMA operand: elements 0..3 from p0 and
// 4..7 from p1.
__device__ __forceinline__ bf16x8 ld_b64x2(const uint16_t* p0, const uint16_t* p1) {
    bf16x4 a = *reinterpret_cast<const bf16x4*>(p0);
    bf16x4 b = *reinterpret_cast<const bf16x4*>(p1);
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

typedef __bf16 bf16v4_t __attribute__((__vector_size__(8)));
typedef __attribute__((address_space(3))) bf16v4_t lds_bf16v4_t;

// LDS tiles hold 64 rows x D BF16 values, row-major without padding, with the
// 16-byte chunks of each row permuted: chunk c of row r lives at chunk
// c ^ swz<D>(r).  The gfx950 LDS has 64 banks of 4 bytes (256 bytes per
// cycle); a 16-byte read is served 16 lanes per cycle and an 8-byte read 32
// lanes per cycle.  Two read patterns hit these tiles: 16-byte reads of one
// chunk from 16 consecutive rows, and transpose reads of 32 bytes (two chunks)
// from 8 consecutive rows.  The swizzle spreads both over 16 distinct 16-byte
// bank groups:
//   d = 64  (128-byte rows, two rows per 256-byte bank line): bits 1..3 of the
//           row pick the chunk within the line for rows of equal parity;
//   d = 128 (256-byte rows): bits 0..3 of the row pick one of 16 chunks.
// The staging writes fill whole 256-byte lines and are conflict free anyway.
// swz<D>(r + 16) == swz<D>(r), so tiles can be addressed 16 rows at a time.
template <int D>
__device__ __forceinline__ int swz(int r) {
    static_assert(D == 64 || D == 128, "head dimension");
    if constexpr (D == 64)
        return (((r >> 1) & 3) << 1) | ((r >> 3) & 1);
    else
        return ((r & 7) << 1) | ((r >> 3) & 1);
}

// Element offset of (row r, column col) in a swizzled tile; col % 4 == 0.
template <int D>
__device__ __forceinline__ int tile_off(int r, int col) {
    return r * D + (((col >> 3) ^ swz<D>(r)) << 3) + (col & 7);
}

// Raw buffer resource over the `bytes` bytes at `base` (stride 0, the gfx9
// data-format word).  The hardware range-checks every buffer load against
// `bytes`: a load at or beyond it returns zero and touches no memory, so tile
// tails need no clamping or masking of addresses.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// 16-byte buffer load at byte offset `off` (zero beyond the resource).
__device__ __forceinline__ u32x4 buf_ld16(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// The same raw buffer resource as four words, for inline assembly.
__device__ __forceinline__ i32x4 buf_desc(const void* base, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    return i32x4{(int32_t)(uint32_t)a, (int32_t)((uint32_t)(a >> 32) & 0xFFFFu), (int32_t)bytes,
                 0x00020000};
}

// 32-bit LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)((__attribute__((address_space(3))) const char*)p);
}

// LDS DMA buffer loads (lane L writes 16 or 4 bytes at M0 + 16 L or M0 + 4 L;
// lanes out of the resource's range write zeros).  They are issued as inline
// assembly so that the compiler's wait-count insertion does not see them: its
// alias tracking of LDS DMA targets is imprecise and would wait for every
// outstanding tile load before each LDS read.  The kernels therefore order
// these loads themselves, with explicit vmcnt waits and barriers (volatile
// assembly keeps its place relative to those).  No memory clobber: nothing
// the compiler reads or writes in LDS overlaps an in-flight DMA target, and a
// clobber would pin every LDS read of the step between the pieces of a fill.
// The s_nop covers the M0-write to LDS-DMA hazard.
__device__ __forceinline__ void lds_dma16(i32x4 desc, uint32_t m0, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(desc));
#else
    (void)desc; (void)m0; (void)voff;
#endif
}
__device__ __forceinline__ void lds_dma4(i32x4 desc, uint32_t m0, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(desc));
#else
    (void)desc; (void)m0; (void)voff;
#endif
}

// Direct global -> LDS staging of one 64-row tile with the gfx950 LDS DMA load
// (buffer_load_dwordx4 ... lds): lane L of a wave writes 16 bytes at
// M0 + 16 L, so each wave call fills a contiguous 1 KB of the swizzled tile
// and every lane loads the global chunk that the swizzle places in its slot.
// No registers or LDS write instructions are involved; completion is tracked
// by vmcnt.  The resource of a call starts at the tile's first row and ends at
// the tensor's last row, so rows at or beyond N are range-checked away: their
// lanes read nothing and write zeros into their LDS slots (measured with an
// in-bounds probe).  The kernels do not rely on that for correctness: every
// probability of a row or key beyond the problem is exactly 0, and the masked
// steps select (not multiply) the operands that meet those rows.
template <int D, int NTHR = kThreads>
struct TileDma {
    static constexpr int NWAVES = NTHR / 64;
    static constexpr int CALLS = kTile * D * 2 / (NTHR * 16);
    uint32_t voff[CALLS];  // byte offset, inside the tile, of this lane's chunk in call k
    uint32_t lds[CALLS];   // byte offset of this wave's 1 KB block (wave-uniform)

    __device__ __forceinline__ void init(int lane, int wave) {
#pragma unroll
        for (int k = 0; k < CALLS; ++k) {
            const int b = (k * NWAVES + wave) * 1024 + 16 * lane;
            const int r = b / (2 * D);
            const int p = (b - r * 2 * D) / 16;
            voff[k] = (uint32_t)(r * 2 * D + ((p ^ swz<D>(r)) * 16));
            lds[k] = (uint32_t)((k * NWAVES + wave) * 1024);
        }
    }
    // Stage rows [row0, row0 + 64) of the [N, D] tensor at `head` into `dst`.
    // With valid == false nothing is read and the slot is filled with zeros
    // (every lane is then out of range), which keeps the number of
    // vector-memory instructions per step fixed.
    __device__ __forceinline__ void load(const uint16_t* head, uint16_t* dst, int row0, int N,
                                         bool valid = true) const {
        const int r0 = valid ? row0 : 0;
        const i32x4 desc =
            buf_desc(head + (size_t)r0 * D, valid ? (uint32_t)(N - r0) * (2 * D) : 0u);
        const uint32_t base = lds_addr(dst);
#pragma unroll
        for (int k = 0; k < CALLS; ++k) lds_dma16(desc, base + lds[k], voff[k]);
    }
    // Call k alone of load(): lets a kernel spread one tile's loads over a step.
    __device__ __forceinline__ void load_call(const uint16_t* head, uint16_t* dst, int row0, int N,
                                              bool valid, int k) const {
        const int r0 = valid ? row0 : 0;
        const i32x4 desc =
            buf_desc(head + (size_t)r0 * D, valid ? (uint32_t)(N - r0) * (2 * D) : 0u);
        lds_dma16(desc, lds_addr(dst) + lds[k], voff[k]);
    }
};

// Per query tile, the key-major pass reads the tile's row statistics from a
// 512-byte block: 64 log2-scaled LSE values, then 64 values of D (FP32).
constexpr int kStatFloats = 2 * kTile;

// LDS DMA of the statistics one wave needs: its 32 query rows (half `qh` of
// the tile) of log2-LSE and of D, 4 bytes per lane, into the 256 bytes at
// `dst` ([32 log2-LSE][32 D]).  A 4-byte LDS DMA writes lane L at M0 + 4 L, so
// the wave's footprint is exactly those 256 bytes.  valid == false writes
// zeros and reads nothing.
__device__ __forceinline__ void stat_dma(const float* tile_stats, float* dst, int lane, int qh,
                                         bool valid) {
    const i32x4 desc = buf_desc(tile_stats, valid ? kStatFloats * 4 : 0);
    const uint32_t row = (uint32_t)(32 * qh + (lane & 31)) + (lane < 32 ? 0u : (uint32_t)kTile);
    lds_dma4(desc, lds_addr(dst), row * 4u);
}

// s_waitcnt with vmcnt <= VM (gfx9 encoding: vmcnt[3:0] | expcnt[6:4] |
// lgkmcnt[11:8] | vmcnt[5:4] at bits 15:14), lgkmcnt = 0, expcnt untouched.
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(VM >= 0 && VM < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | ((VM >> 4) << 14));
}

// Transposed MFMA operand read straight from a row-major LDS tile X[k][n]
// with the gfx950 LDS transpose load ds_read_b64_tr_b16.  Within each 16-lane
// group, that instruction hands lane j element j of the 4 x 16 block formed by
// the 8-byte reads of lanes 4r+q (row r, columns 4q..4q+3).  Addressing rows
// k0+4g+r and columns n0+4q therefore gives lane (c16, g) the values
// X[k0 + 4g + r][n0 + c16], r = 0..3; a second read 16 rows further down fills
// elements 4..7.  This is the k-layout {4g+r, 16+4g+r} that the 16x16
// accumulator of the preceding product leaves in each lane.
template <int D>
__device__ __forceinline__ bf16x8 ld_tr_operand(const uint16_t* X, int k0, int n0, int c16,
                                                int g) {
    const int row = k0 + 4 * g + (c16 >> 2);
    const uint16_t* p0 = X + tile_off<D>(row, n0 + 4 * (c16 & 3));
    const uint16_t* p1 = p0 + 16 * D;  // row + 16 has the same swizzle
    const bf16x4 a =
        __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16v4_t*)p0));
    const bf16x4 b =
        __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16v4_t*)p1));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ __bf16 to_bf16(float x) { return static_cast<__bf16>(x); }
__device__ __forceinline__ float bf16_to_f32(__bf16 x) { return static_cast<float>(x); }

__device__ __forceinline__ uint16_t bf16_bits(float x) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

// Store 4 floats as 4 consecutive BF16 values (8 bytes).
__device__ __forceinline__ void st_bf16x4(uint16_t* p, float a, float b, float c, float d) {
    bf16x4 v;
    v[0] = to_bf16(a); v[1] = to_bf16(b); v[2] = to_bf16(c); v[3] = to_bf16(d);
    *reinterpret_cast<bf16x4*>(p) = v;
}

// BF16 halves of a packed 32-bit word, widened exactly to FP32.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// 16-byte load of row `row` at column `col` of a [N, D] tensor whose buffer
// resource `r` covers exactly its N rows: rows at or beyond N read as zero.
template <int D>
__device__ __forceinline__ u32x4 ld_row16(rsrc_t r, int row, int col) {
    return buf_ld16(r, (uint32_t)(row * D + col) * 2u);
}

// MFMA A operand whose row 0 is all ones and rows 1..15 zero: multiplying it
// into a B operand gives the column sums of B in accumulator row 0.
__device__ __forceinline__ bf16x8 ones_row0(int c16) {
    const __bf16 v = (c16 == 0) ? (__bf16)1.0f : (__bf16)0.0f;
    bf16x8 a;
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = v;
    return a;
}

// Reductions over the four 16-lane rows of a wave (lanes c16, c16 + 16,
// c16 + 32, c16 + 48), with the gfx950 lane-swap instructions instead of an
// LDS round trip.  v_permlane16_swap on two copies of v leaves rows (0, 0, 2, 2)
// in one copy and (1, 1, 3, 3) in the other; v_permlane32_swap leaves the low
// and the high half.  Combining the two copies therefore gives every lane the
// pairwise result (x ^ 16, then x ^ 32), bitwise the same in both partners
// because max and + are commutative.
__device__ __forceinline__ float xor_max(float v) {
    const uint32_t u = __float_as_uint(v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const uint32_t w = __float_as_uint(v);
    const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float xor_sum(float v) {
    const uint32_t u = __float_as_uint(v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const uint32_t w = __float_as_uint(v);
    const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Workgroup -> (batch*head, tile).  Workgroups are dispatched round-robin over
// the 8 XCDs (each with its own L2), and within an XCD to whichever slots free
// up first.  When B*H is a multiple of 8, XCD x owns heads [x*BH/8, (x+1)*BH/8)
// so one head's tiles share an L2.  Those heads are taken in groups of hg,
// just enough heads for kGroupTiles workgroups (about twice the workgroups an
// XCD holds at once), one group after the other: the tiles in flight then
// stream the data of one or two heads, not of every head of the XCD (which
// would not fit in its L2 at long sequences).  Within a group the order is
// rank-major: every head's heaviest tile, then every head's next heaviest,
// ... , which makes the hardware's in-order dispatch a longest-first greedy
// schedule for any number of resident workgroups.  heavy_high selects which
// end is heavy: the query-major causal kernels' last tiles do the most work,
// the key-major kernels' first tiles do.
//
// snake_rounds: an XCD places its i-th workgroup on compute unit i mod 32
// while it has free slots, so the first `resident` x 32 workgroups of an XCD
// (resident = workgroups a unit holds) are placed before any finishes.
// Reversing every other block of 32 of those positions deals the heavy-first
// list out like a snake draft: compute unit p gets list positions p, 63 - p,
// 64 + p, 127 - p, ..., about the same total work on every unit.  This pays
// when the resident set holds most of the grid (the d = 64 forward, 4 per
// unit); later workgroups keep the longest-first order, which the in-order
// dispatch balances by itself (with 2 per unit the backward passes measured
// slower with the snake).
constexpr int kGroupTiles = 128;
constexpr int kXcdCUs = 32;  // compute units per XCD
__device__ __forceinline__ void map_block(int bid, int BH, int T, bool heavy_high, int* bh,
                                          int* tile, int snake_rounds = 0) {
    int heads = BH, base = 0, li = bid;
    if ((BH & 7) == 0) {
        heads = BH >> 3;
        base = (bid & 7) * heads;
        li = bid >> 3;
        const int q = li / kXcdCUs, p = li - q * kXcdCUs;
        if ((q & 1) && q < snake_rounds && q < (heads * T) / kXcdCUs)
            li = q * kXcdCUs + (kXcdCUs - 1 - p);
    }
    const int hg = min(heads, max(1, (kGroupTiles + T - 1) / T));
    const int group = li / (hg * T);
    const int first = group * hg;
    const int gs = min(hg, heads - first);  // the last group may be smaller
    const int within = li - group * hg * T;
    const int rank = within / gs;
    *bh = base + first + (within - rank * gs);
    *tile = heavy_high ? (T - 1 - rank) : rank;
}

// Rows of one attention problem (a query head of one sequence) and its query
// and key counts.  Dense batches ([B, H, N, d], cu == nullptr): query head
// bh = b * Hq + h starts at row bh * N of Q and reads key/value head bh / G;
// nq = nk = N.  Packed sequences (query-side tensors [H, total, d], key-side
// [H, total_k, d]): bh = s * Hq + h is head h over queries [cu[s], cu[s + 1])
// and keys [cu_k[s], cu_k[s + 1]); the offsets are clamped to the tensors and
// the counts to the longest runs, so malformed offsets cannot address rows
// outside the tensors.  With causal masking query i sees key j iff
// j <= i + (nk - nq): the diagonal is aligned at the last query and key.
struct SeqRows {
    size_t q0;   // first row of the query-head tensors (Q, O, dO, dQ; LSE, row statistics)
    size_t kv0;  // first row of the key/value-head tensors (K, V, dK, dV)
    size_t p0;   // first row of this query head's key-side FP32 partials (grouped heads)
    int nq;      // queries of this problem
    int nk;      // keys of this problem
};
__device__ __forceinline__ SeqRows seq_rows(const int* cu, const int* cu_k, int bh, int Nq_max,
                                            int Nk_max, int G, int Hq, int total, int total_k) {
    if (cu == nullptr)
        return {(size_t)bh * Nq_max, (size_t)(bh / G) * Nq_max, (size_t)bh * Nq_max, Nq_max,
                Nq_max};
    const int s = bh / Hq, h = bh - s * Hq;
    const int a = min(max(cu[s], 0), total);
    const int b = min(max(cu[s + 1], a), total);
    const int ak = min(max(cu_k[s], 0), total_k);
    const int bk = min(max(cu_k[s + 1], ak), total_k);
    return {(size_t)h * total + a, (size_t)(h / G) * total_k + ak, (size_t)h * total_k + ak,
            min(b - a, Nq_max), min(bk - ak, Nk_max)};
}

// Floor division by a positive divisor, also for negative numerators.
__device__ __forceinline__ int floor_div(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// Key tiles of a 64-query tile: keys [0, 64 * nkv) hold every key a query of
// the tile can see, and tiles [nplain, nkv) need masks (at most two: the
// causal diagonal crosses at most two key tiles, and the key tail).
struct KeyRange {
    int nkv, nplain;
};
__device__ __forceinline__ KeyRange key_range(int qtile, int Nk, int off, int causal) {
    const int kv_end = causal ? min(max((qtile + 1) * kTile + off, 0), Nk) : Nk;
    const int nkv = (kv_end + kTile - 1) / kTile;
    // fully visible tiles: every key <= the first query's last visible key, and
    // no key beyond Nk
    const int nfull = causal ? floor_div(qtile * kTile + off + 1, kTile) : Nk / kTile;
    return {nkv, max(0, min(min(nfull, Nk / kTile), nkv))};
}

// Target waves per SIMD of each MFMA kernel (build-time tuning constants).
#ifndef GPA_FWD_OCC
#define GPA_FWD_OCC 2
#endif
#ifndef GPA_FWD16_OCC
#define GPA_FWD16_OCC 4
#endif
#ifndef GPA_DQ_OCC64
#define GPA_DQ_OCC64 2
#endif
#ifndef GPA_DKDV_OCC64
#define GPA_DKDV_OCC64 2
#endif

}  // namespace gpa
