// Device-side helpers shared by the gfx950 kernels of libgpa.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gpa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// FP32 log2(e), rounded to FP32.
constexpr float kLog2e = 1.44269504088896340736f;

// Tile geometry shared by the MFMA kernels.  A wave owns 16 rows of its
// operand (queries in the forward and the query-major backward, keys in the
// key-major backward); a workgroup has 4 waves.
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kTile = 64;  // rows per workgroup tile and per streamed tile

// LDS row pitches (in 16-bit elements).  Row-major tiles are read 16 bytes per
// lane by 16 lanes on different rows: a pitch of d+8 elements (d*2+16 bytes)
// puts consecutive rows 4 banks apart.  Transposed tiles are read 8 bytes per
// lane on 16 different rows: a pitch of 64+4 elements (136 bytes) puts them 2
// banks apart.
template <int D> struct Pitch {
    static constexpr int row = D + 8;
    static constexpr int tr = kTile + 4;
};

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

// Transposed MFMA operand read straight from a row-major LDS tile X[k][n]
// (pitch P elements) with the gfx950 LDS transpose load ds_read_b64_tr_b16.
// Within each 16-lane group, that instruction hands lane j element j of the
// 4 x 16 block formed by the 8-byte reads of lanes 4r+q (row r, columns
// 4q..4q+3).  Addressing rows k0+4g+r and columns n0+4q therefore gives lane
// (c16, g) the values X[k0 + 4g + r][n0 + c16], r = 0..3; a second read 16 rows
// further down fills elements 4..7.  This is the k-layout {4g+r, 16+4g+r} that
// the 16x16 accumulator of the preceding product leaves in each lane.
__device__ __forceinline__ bf16x8 ld_tr_operand(const uint16_t* X, int P, int k0, int n0,
                                                int c16, int g) {
    const uint16_t* p0 = X + (k0 + 4 * g + (c16 >> 2)) * P + n0 + 4 * (c16 & 3);
    const uint16_t* p1 = p0 + 16 * P;
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

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// BF16 halves of a packed 32-bit word, widened exactly to FP32.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// 16-byte global load of row `row` (clamped into [0, N)) at column `col`;
// rows at or beyond N read as zero.  Branch-free and always in bounds.
__device__ __forceinline__ u32x4 ld_row16(const uint16_t* base, int row, int N, int D, int col) {
    const int r = row < N ? row : N - 1;
    u32x4 w = *reinterpret_cast<const u32x4*>(base + (size_t)r * D + col);
    const uint32_t keep = row < N ? 0xFFFFFFFFu : 0u;
    w[0] &= keep; w[1] &= keep; w[2] &= keep; w[3] &= keep;
    return w;
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

__device__ __forceinline__ float xor_max(float v) {
    v = fmaxf(v, __shfl_xor(v, 16));
    v = fmaxf(v, __shfl_xor(v, 32));
    return v;
}

__device__ __forceinline__ float xor_sum(float v) {
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

// Workgroup -> (batch*head, tile).  Workgroups are dispatched round-robin over
// the 8 XCDs (each with its own L2), so when the grid divides evenly, XCD x is
// given a contiguous range of (head, tile) pairs: the tiles of one head share
// that XCD's L2.  Within a head, tiles go out in the order given by
// heavy_first_desc (descending tile index for the query-major causal kernels,
// whose last tiles have the most work; ascending for the key-major ones).
__device__ __forceinline__ void map_block(int bid, int BH, int T, bool heavy_first_desc,
                                          int* bh, int* tile) {
    const int nwg = BH * T;
    int linear = bid;
    if ((nwg & 7) == 0) {
        const int per = nwg >> 3;
        linear = (bid & 7) * per + (bid >> 3);
    }
    *bh = linear / T;
    const int t = linear - (*bh) * T;
    *tile = heavy_first_desc ? (T - 1 - t) : t;
}

}  // namespace gpa
