// Chunk summary (section "EVA Attention": after eq. (eva_normalization), one
// random-feature sample per chunk makes the chunk's value independent of the
// query, so it is computed once per chunk; the concrete form used here is the
// mean key and the value weighted by softmax(mean-key . key / sqrt(d))).
//
//   khat = (1/C) sum_j k_j
//   a_j  = khat . k_j / sqrt(d)           (kept in log2 units: * log2(e))
//   vhat = sum_j exp(a_j - max a) v_j / sum_j exp(a_j - max a)
//
// One 256-thread workgroup computes one chunk.  Each key/value row is split
// over TPR = D/8 threads holding 8 features each; the workgroup covers
// RPS = 256/TPR rows per step.  Pass 1 sums the keys (loads straight from
// HBM, 16 B per lane), pass 2 re-reads the keys (cache hits) for the scores,
// pass 3 streams the values.  All arithmetic in fp32.
#pragma once

#include "eva_device.hpp"

namespace eva {

constexpr int kSummaryThreads = 256;

// Row-major source: rows of D elements, row r of the chunk at base + r * D.
template <int D, typename T>
struct RowMajorChunk {
    const T* k;
    const T* v;
    __device__ void load8(const T* base, int r, int cc, float out[8]) const {
        const T* p = base + (size_t)r * D + cc * 8;
        if constexpr (sizeof(T) == 2) {
            u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                out[2 * i] = bf16_lo(w[i]);
                out[2 * i + 1] = bf16_hi(w[i]);
            }
        } else {
            floatx4 a = *reinterpret_cast<const floatx4*>(p);
            floatx4 b = *reinterpret_cast<const floatx4*>(p + 4);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                out[i] = a[i];
                out[4 + i] = b[i];
            }
        }
    }
    __device__ void load_k(int r, int cc, float out[8]) const { load8(k, r, cc, out); }
    __device__ void load_v(int r, int cc, float out[8]) const { load8(v, r, cc, out); }
};

// Cache ring source: row r of the chunk is position pos0 + r, stored in slot
// (pos0 + r) mod R; keys row-major [R][D], values transposed per 8-slot tile
// [R/8][D][8] (vt_index).
template <int D, typename T>
struct RingChunk {
    const T* k_ring;   // this (b, g): [R][D]
    const T* vt_ring;  // this (b, g): [R/8][D][8]
    long long pos0;
    int R;
    __device__ int slot(int r) const { return (int)((pos0 + r) % R); }
    __device__ void load_k(int r, int cc, float out[8]) const {
        const T* p = k_ring + (size_t)slot(r) * D + cc * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = to_f32(p[i]);
    }
    __device__ void load_v(int r, int cc, float out[8]) const {
        int s = slot(r);
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = to_f32(vt_ring[vt_index<D>(cc * 8 + i, s)]);
    }
};

// A chunk completed by the token being appended: rows 0 .. C-2 are still in
// the ring (positions pos0 .. pos0 + C - 2), row C-1 is the new token, read
// from the caller's [D] input vectors (it is not in the ring yet).
template <int D, typename T>
struct RingChunkPlusNew {
    RingChunk<D, T> ring;
    const T* k_new;  // this (b, g): [D]
    const T* v_new;
    int last;        // C - 1
    __device__ void load_k(int r, int cc, float out[8]) const {
        if (r == last) {
#pragma unroll
            for (int i = 0; i < 8; ++i) out[i] = to_f32(k_new[cc * 8 + i]);
        } else {
            ring.load_k(r, cc, out);
        }
    }
    __device__ void load_v(int r, int cc, float out[8]) const {
        if (r == last) {
#pragma unroll
            for (int i = 0; i < 8; ++i) out[i] = to_f32(v_new[cc * 8 + i]);
        } else {
            ring.load_v(r, cc, out);
        }
    }
};

// Reduce an 8-vector over all threads that share the same feature chunk cc
// (lanes l, l^TPR, l^2TPR, ... inside the wave, then the waves through LDS).
// Returns the total in the threads of wave 0 whose row index is 0 (t < TPR),
// and leaves it in red[cc*8 + i] for everyone after the final barrier.
template <int TPR>
__device__ void reduce_rows8(float v[8], float* red /* [4][TPR*8] */) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
        for (int off = TPR; off < 64; off <<= 1) v[i] += __shfl_xor(v[i], off, 64);
    }
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    if (lane < TPR) {
#pragma unroll
        for (int i = 0; i < 8; ++i) red[wave * TPR * 8 + lane * 8 + i] = v[i];
    }
    __syncthreads();
    if (t < TPR * 8) {
        float s = red[t] + red[TPR * 8 + t] + red[2 * TPR * 8 + t] + red[3 * TPR * 8 + t];
        red[4 * TPR * 8 + t] = s;
    }
    __syncthreads();
    const int cc = t % TPR;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = red[4 * TPR * 8 + cc * 8 + i];
    __syncthreads();
}

__device__ __forceinline__ float block_max(float x, float* red) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
    const int t = threadIdx.x;
    if ((t & 63) == 0) red[t >> 6] = x;
    __syncthreads();
    float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    return m;
}

// Logit weight vector of one thread's 8 features.  Deterministic summaries:
// the mean key (logit khat . k).  Stochastic random-feature summaries
// (one sample omega = mean scaled key + lambda * clip(eps, -1, 1) per chunk,
// feature map exp(omega . x - |x|^2 / 2) on the scaled keys x = k / d^(1/4)):
// the logit times sqrt(d) is k . (khat + lambda d^(1/4) clip(eps) - k / 2),
// so the weight vector is khat + rf_scale * clip(eps) and the row adds -k/2.
struct RfNoise {
    const float* eps;  // this thread's 8 noise values (nullptr: deterministic)
    float scale;       // lambda * d^(1/4)
};

// Computes the summary of one chunk of C rows.  `logits` holds C floats of
// LDS, `red` 5*TPR*8 floats of LDS.  Results: khat[8], vhat[8] for this
// thread's feature chunk cc = threadIdx.x % TPR (valid in every thread).
template <int D, bool RF = false, typename Src>
__device__ void chunk_summary(const Src& src, int C, float* logits, float* red, float khat[8], float vhat[8],
                              RfNoise rf = {nullptr, 0.f}) {
    constexpr int TPR = D / 8;
    constexpr int RPS = kSummaryThreads / TPR;
    const int t = threadIdx.x;
    const int cc = t % TPR;
    const int r0 = t / TPR;

    // pass 1: mean key
    float ks[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int r = r0; r < C; r += RPS) {
        float k[8];
        src.load_k(r, cc, k);
#pragma unroll
        for (int i = 0; i < 8; ++i) ks[i] += k[i];
    }
    reduce_rows8<TPR>(ks, red);
    const float invC = 1.0f / (float)C;
#pragma unroll
    for (int i = 0; i < 8; ++i) khat[i] = ks[i] * invC;

    // pass 2: scores a_j (log2 units) into LDS, running max
    const float sc = kLog2e * rsqrtf((float)D);
    float w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = RF ? khat[i] + rf.scale * fminf(fmaxf(rf.eps[i], -1.f), 1.f) : khat[i];
    float amax = -INFINITY;
    for (int r = r0; r < C; r += RPS) {
        float k[8];
        src.load_k(r, cc, k);
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += (RF ? w[i] - 0.5f * k[i] : w[i]) * k[i];
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) s += __shfl_xor(s, off, 64);
        s *= sc;
        if (cc == 0) logits[r] = s;
        amax = fmaxf(amax, s);
    }
    amax = block_max(amax, red);  // also orders the logits writes before the reads

    // pass 3: softmax-weighted values
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
    for (int r = r0; r < C; r += RPS) {
        float v[8];
        src.load_v(r, cc, v);
        float p = fast_exp2(logits[r] - amax);
        psum += p;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += p * v[i];
    }
    // psum: every thread of a row group summed the same rows; reduce over rows
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) psum += __shfl_xor(psum, off, 64);
    if ((t & 63) == 0) red[5 * TPR * 8 + (t >> 6)] = psum;
    __syncthreads();
    const float den = red[5 * TPR * 8] + red[5 * TPR * 8 + 1] + red[5 * TPR * 8 + 2] + red[5 * TPR * 8 + 3];
    __syncthreads();
    reduce_rows8<TPR>(acc, red);
    const float inv = 1.0f / den;
#pragma unroll
    for (int i = 0; i < 8; ++i) vhat[i] = acc[i] * inv;
}

template <int D>
constexpr int summary_red_floats() { return 5 * (D / 8) * 8 + 4; }

}  // namespace eva
