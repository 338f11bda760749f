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
