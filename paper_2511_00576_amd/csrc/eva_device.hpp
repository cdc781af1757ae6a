// Device-side building blocks shared by the EVA kernels (gfx950 / CDNA4).
//
// Matrix-core operand layouts used throughout (wave of 64 lanes, lane l,
// lane group g = l / 16, column c = l % 16):
//   v_mfma_f32_16x16x32_bf16  A[16 x 32]: lane holds A[c][8g .. 8g+7]
//                             B[32 x 16]: lane holds B[8g .. 8g+7][c]
//                             D[16 x 16]: lane holds D[4g .. 4g+3][c]
//   v_mfma_f32_16x16x4_f32    A[16 x 4]:  lane holds A[c][g]
//                             B[4 x 16]:  lane holds B[g][c]
//                             D as above.
// The contraction index may be permuted freely as long as A and B agree.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eva {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 with round-to-nearest-even (hardware conversion on gfx950).
__device__ __forceinline__ bf16 to_bf16(float x) { return (bf16)x; }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16 a = to_bf16(lo), b = to_bf16(hi);
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return to_bf16(x); }

__device__ __forceinline__ floatx4 mfma_bf16(const bf16x8& a, const bf16x8& b, const floatx4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma_f32(float a, float b, const floatx4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Reductions across the four 16-lane groups (lanes l, l^16, l^32, l^48):
// v_permlane16_swap / v_permlane32_swap exchange halves of the wave in one
// VALU op each, no LDS traffic.
__device__ __forceinline__ float xgroup_max(float x) {
    uint32_t u = __float_as_uint(x);
    auto s16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    float y = fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
    uint32_t v = __float_as_uint(y);
    auto s32 = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
}
__device__ __forceinline__ float xgroup_sum(float x) {
    uint32_t u = __float_as_uint(x);
    auto s16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    float y = __uint_as_float(s16[0]) + __uint_as_float(s16[1]);
    uint32_t v = __float_as_uint(y);
    auto s32 = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __uint_as_float(s32[0]) + __uint_as_float(s32[1]);
}

// LDS transposing read: each lane of a 16-lane group passes the address of 4
// consecutive 16-bit elements; lanes 4j..4j+3 together name row j (16
// elements).  Lane i of the group receives element i of rows 0..3.
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
__device__ __forceinline__ shortx4 lds_read_tr16(const bf16* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(p));
}

// Transposed value arrays of the decode cache are tiled by 8 rows: row (slot
// or summary index) r, feature f lives at element
//   (r / 8) * 8 * D + f * 8 + r % 8,
// so a tile is one contiguous [D][8] block, each feature's 8 slots one
// 16-byte piece (one matrix-core operand fragment), and 32 consecutive rows
// (the decode's unit) 4 consecutive tiles.  Short tiles keep the write of a
// single appended row to D / 8 cache lines (D / 2 with 32-row tiles).
constexpr int kVtTile = 8;
template <int D>
__host__ __device__ __forceinline__ size_t vt_index(int f, int r) {
    return (size_t)(r >> 3) * (kVtTile * D) + (size_t)f * kVtTile + (r & 7);
}

// Counter-based normal draws for the stochastic summaries, so that the draw
// of chunk c of sequence-head s is the same wherever its summary is built.
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds over a
// 128-bit counter with a 64-bit key; a round takes the 64-bit products of
// counter words 0 and 2 with two fixed multipliers, swaps their halves in and
// mixes in the key, which advances by two fixed increments between rounds.
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t m0 = 0xD2511F53u, m1 = 0xCD9E8D57u;
        const uint32_t hi0 = __umulhi(m0, c[0]), lo0 = m0 * c[0];
        const uint32_t hi1 = __umulhi(m1, c[2]), lo1 = m1 * c[2];
        const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

// Normals for features 4i .. 4i+3 of chunk `chunk` of sequence-head `seq`:
// Philox block at counter (i, chunk, seq, 0), key = the seed's two words;
// each word pair (x, y) gives two normals by the Box-Muller transform on the
// 24-bit uniforms u = ((x >> 8) + 1/2) 2^-24, v = ((y >> 8) + 1/2) 2^-24:
// sqrt(-2 ln u) (cos 2 pi v, sin 2 pi v).
__device__ __forceinline__ void rf_normals4(unsigned long long seed, uint32_t i, uint32_t chunk, uint32_t seq,
                                            float out[4]) {
    uint32_t c[4] = {i, chunk, seq, 0u};
    philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const float u = ((float)(c[2 * h] >> 8) + 0.5f) * 5.9604644775390625e-8f;  // 2^-24
        const float v = ((float)(c[2 * h + 1] >> 8) + 0.5f) * 5.9604644775390625e-8f;
        const float r = sqrtf(-2.f * logf(u));
        float sn, cs;
        sincosf(6.283185307179586f * v, &sn, &cs);
        out[2 * h] = r * cs;
        out[2 * h + 1] = r * sn;
    }
}

// Window variants (values of the ABI's eva_window).  Row n attends the exact
// keys [win_lo(n), win_hi(n)] and the summaries of the complete chunks
// c < sum_lo(n) (those ending at or before win_lo) and, non-causal only,
// c >= sum_hi(n) (those starting after win_hi).  All four are non-decreasing
// in n.
constexpr int kWinSliding = 0;       // [n-W+1, n]
constexpr int kWinChunkAligned = 1;  // sliding start rounded down to its chunk
constexpr int kWinBlocked = 2;       // [floor(n/W) W, n]
constexpr int kWinNonCausal = 3;     // the whole block [floor(n/W) W, +W)

template <int VAR>
__device__ __forceinline__ int win_lo(int n, int W, int C) {
    if constexpr (VAR == kWinSliding) return max(0, n - W + 1);
    if constexpr (VAR == kWinChunkAligned) return (max(0, n - W + 1) / C) * C;
    return (n / W) * W;
}
template <int VAR>
__device__ __forceinline__ int win_hi(int n, int W, int L) {
    if constexpr (VAR == kWinNonCausal) return min(L, (n / W) * W + W) - 1;
    return n;
}
template <int VAR>
__device__ __forceinline__ int sum_lo(int n, int W, int C) {
    return win_lo<VAR>(n, W, C) / C;
}
template <int VAR>
__device__ __forceinline__ int sum_hi(int n, int W, int C, int L) {
    return win_hi<VAR>(n, W, L) / C + 1;
}

// Runtime-variant forms (decode geometry).
__device__ __forceinline__ int win_lo_rt(int variant, int n, int W, int C) {
    switch (variant) {
        case kWinChunkAligned: return win_lo<kWinChunkAligned>(n, W, C);
        case kWinBlocked: return win_lo<kWinBlocked>(n, W, C);
        default: return win_lo<kWinSliding>(n, W, C);
    }
}

}  // namespace eva
