// Chunk-summary kernel for the prefill path: K, V row-major [BH][L][D] ->
// Ks, Vs row-major [BH][L / C][D].  One workgroup per chunk; HBM bound
// (reads every key and value once, writes two rows per chunk).
#include "eva_kernels.hpp"
#include "summary.hpp"

namespace eva {

namespace {

// eps (RF only): fp32 [BH][n_chunks][D], one noise draw per chunk;
// rf_scale = lambda * d^(1/4).
template <int D, typename T, bool RF>
__global__ __launch_bounds__(kSummaryThreads) void summary_kernel(const T* __restrict__ K, const T* __restrict__ V,
                                                                  T* __restrict__ Ks, T* __restrict__ Vs, int L,
                                                                  int C, int n_chunks, const float* __restrict__ eps,
                                                                  float rf_scale) {
    extern __shared__ float smem[];
    constexpr int TPR = D / 8;
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const size_t row0 = bg * (size_t)L + (size_t)chunk * C;
    RowMajorChunk<D, T> src{K + row0 * D, V + row0 * D};
    float kh[8], vh[8];
    const RfNoise rf{RF ? eps + (bg * n_chunks + chunk) * D + (threadIdx.x % TPR) * 8 : nullptr, rf_scale};
    chunk_summary<D, RF>(src, C, smem, smem + C, kh, vh, rf);
    const int t = threadIdx.x;
    if (t < TPR) {
        const size_t out = (bg * n_chunks + chunk) * D + t * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            Ks[out + i] = from_f32<T>(kh[i]);
            Vs[out + i] = from_f32<T>(vh[i]);
        }
    }
}

// Register-resident variant for chunks of exactly ROWS * RPS rows: every
// thread requests all of its key and value rows up front (one memory latency
// per chunk instead of one per pass), keeps them in registers, and the three
// passes of the summary run on those registers.
template <int D, typename T, int ROWS, bool RF>
__global__ __launch_bounds__(kSummaryThreads) void summary_kernel_reg(const T* __restrict__ K, const T* __restrict__ V,
                                                                      T* __restrict__ Ks, T* __restrict__ Vs, int L,
                                                                      int n_chunks, const float* __restrict__ eps,
                                                                      float rf_scale) {
    constexpr int TPR = D / 8;
    constexpr int RPS = kSummaryThreads / TPR;
    constexpr int C = ROWS * RPS;
    constexpr int VW = sizeof(T) == 2 ? 1 : 2;  // 16-B words per 8 elements
    __shared__ float red[summary_red_floats<D>()];
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const int t = threadIdx.x, cc = t % TPR, r0 = t / TPR;
    const size_t row0 = bg * (size_t)L + (size_t)chunk * C;
    const T* kp = K + (row0 + r0) * D + cc * 8;
    const T* vp = V + (row0 + r0) * D + cc * 8;

    u32x4 kw[ROWS][VW], vw[ROWS][VW];
    floatx4 ew[2];
    if constexpr (RF) {
        const float* ep = eps + (bg * n_chunks + chunk) * D + cc * 8;
        ew[0] = *reinterpret_cast<const floatx4*>(ep);
        ew[1] = *reinterpret_cast<const floatx4*>(ep + 4);
    }
    // every row is read exactly once: non-temporal loads keep the stream from
    // displacing cached data (measured: 94 -> 84 us on the LLM workload, and
    // the attention kernel after it runs faster too)
#pragma unroll
    for (int i = 0; i < ROWS; ++i)
#pragma unroll
        for (int w = 0; w < VW; ++w) {
            kw[i][w] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + (size_t)i * RPS * D + w * (8 / VW)));
            vw[i][w] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vp + (size_t)i * RPS * D + w * (8 / VW)));
        }
    auto unpack = [&](const u32x4 (&x)[VW], float out[8]) {
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                out[2 * e] = bf16_lo(x[0][e]);
                out[2 * e + 1] = bf16_hi(x[0][e]);
            }
        } else {
#pragma unroll
            for (int w = 0; w < VW; ++w)
#pragma unroll
                for (int e = 0; e < 4; ++e) out[w * 4 + e] = __uint_as_float(x[w][e]);
        }
    };

    // pass 1: mean key
    float kh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
#pragma unroll
        for (int e = 0; e < 8; ++e) kh[e] += k[e];
    }
    reduce_rows8<TPR>(kh, red);
#pragma unroll
    for (int e = 0; e < 8; ++e) kh[e] *= 1.0f / (float)C;

    // pass 2: scores (log2 units); the TPR threads of a row hold its full
    // score.  Weight vector as in chunk_summary (RfNoise).
    const float sc = kLog2e * rsqrtf((float)D);
    float w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        w[e] = RF ? kh[e] + rf_scale * fminf(fmaxf(ew[e >> 2][e & 3], -1.f), 1.f) : kh[e];
    float s[ROWS];
    float amax = -INFINITY;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) x += (RF ? w[e] - 0.5f * k[e] : w[e]) * k[e];
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) x += __shfl_xor(x, off, 64);
        s[i] = x * sc;
        amax = fmaxf(amax, s[i]);
    }
    amax = block_max(amax, red);

    // pass 3: softmax-weighted values
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float v[8];
        unpack(vw[i], v);
        const float p = fast_exp2(s[i] - amax);
        psum += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += p * v[e];
    }
    // psum: the threads of a row group summed the same rows; reduce over rows
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) psum += __shfl_xor(psum, off, 64);
    if ((t & 63) == 0) red[5 * TPR * 8 + (t >> 6)] = psum;
    __syncthreads();
    const float den = red[5 * TPR * 8] + red[5 * TPR * 8 + 1] + red[5 * TPR * 8 + 2] + red[5 * TPR * 8 + 3];
    __syncthreads();
    reduce_rows8<TPR>(acc, red);
    if (t < TPR) {
        const float inv = 1.0f / den;
        const size_t out = (bg * n_chunks + chunk) * D + t * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            Ks[out + e] = from_f32<T>(kh[e]);
            Vs[out + e] = from_f32<T>(acc[e] * inv);
        }
    }
}

// One-wave variant (bf16): 64 threads per chunk, ROWS rows per thread, every
// reduction inside the wave (shuffles only: no LDS, no barrier).
template <int D, int ROWS, bool RF>
__global__ __launch_bounds__(64) void summary_kernel_wave(const bf16* __restrict__ K, const bf16* __restrict__ V,
                                                          bf16* __restrict__ Ks, bf16* __restrict__ Vs, int L,
                                                          int n_chunks, const float* __restrict__ eps,
                                                          float rf_scale) {
    constexpr int TPR = D / 8;
    constexpr int RPS = 64 / TPR;
    constexpr int C = ROWS * RPS;
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const int t = threadIdx.x, cc = t % TPR, r0 = t / TPR;
    const size_t row0 = bg * (size_t)L + (size_t)chunk * C;
    const bf16* kp = K + (row0 + r0) * D + cc * 8;
    const bf16* vp = V + (row0 + r0) * D + cc * 8;
    u32x4 kw[ROWS], vw[ROWS];
    floatx4 ew[2];
    if constexpr (RF) {
        const float* ep = eps + (bg * n_chunks + chunk) * D + cc * 8;
        ew[0] = *reinterpret_cast<const floatx4*>(ep);
        ew[1] = *reinterpret_cast<const floatx4*>(ep + 4);
    }
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        kw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + (size_t)i * RPS * D));
        vw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vp + (size_t)i * RPS * D));
    }
    auto unpack = [](const u32x4& x, float out[8]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[2 * e] = bf16_lo(x[e]);
            out[2 * e + 1] = bf16_hi(x[e]);
        }
    };
    // sum over the lanes holding the same features (the row groups)
    auto rows_sum = [](float& x) {
#pragma unroll
        for (int off = TPR; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
    };
    float kh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
#pragma unroll
        for (int e = 0; e < 8; ++e) kh[e] += k[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        rows_sum(kh[e]);
        kh[e] *= 1.0f / (float)C;
    }
    const float sc = kLog2e * rsqrtf((float)D);
    float w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        w[e] = RF ? kh[e] + rf_scale * fminf(fmaxf(ew[e >> 2][e & 3], -1.f), 1.f) : kh[e];
    float s[ROWS];
    float amax = -INFINITY;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) x += (RF ? w[e] - 0.5f * k[e] : w[e]) * k[e];
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) x += __shfl_xor(x, off, 64);
        s[i] = x * sc;
        amax = fmaxf(amax, s[i]);
    }
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float v[8];
        unpack(vw[i], v);
        const float p = fast_exp2(s[i] - amax);
        psum += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += p * v[e];
    }
    rows_sum(psum);
#pragma unroll
    for (int e = 0; e < 8; ++e) rows_sum(acc[e]);
    if (t < TPR) {
        const float inv = 1.0f / psum;
        const size_t out = (bg * n_chunks + chunk) * D + t * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            Ks[out + e] = to_bf16(kh[e]);
            Vs[out + e] = to_bf16(acc[e] * inv);
        }
    }
}

template <int D, typename T, bool RF>
hipError_t launch_summaries_impl(const void* K, const void* V, void* Ks, void* Vs, int BH, int L, int C,
                                 const float* eps, float rf_scale, hipStream_t stream) {
    const int n_chunks = L / C;
    if (n_chunks == 0) return hipSuccess;
    constexpr int RPS = kSummaryThreads / (D / 8);
    const T* k = static_cast<const T*>(K);
    const T* v = static_cast<const T*>(V);
    T* ks = static_cast<T*>(Ks);
    T* vs = static_cast<T*>(Vs);
    if constexpr (sizeof(T) == 2) {
        // one wave per chunk when the chunk is 4, 8 or 16 rows per thread of it
        constexpr int RPW = 64 / (D / 8);
        const dim3 grid(n_chunks, BH);
        switch (C % RPW == 0 ? C / RPW : 0) {
            case 4:
                hipLaunchKernelGGL((summary_kernel_wave<D, 4, RF>), grid, dim3(64), 0, stream, k, v, ks, vs, L, n_chunks,
                                   eps, rf_scale);
                return hipGetLastError();
            case 8:
                hipLaunchKernelGGL((summary_kernel_wave<D, 8, RF>), grid, dim3(64), 0, stream, k, v, ks, vs, L, n_chunks,
                                   eps, rf_scale);
                return hipGetLastError();
            case 16:
                hipLaunchKernelGGL((summary_kernel_wave<D, 16, RF>), grid, dim3(64), 0, stream, k, v, ks, vs, L,
                                   n_chunks, eps, rf_scale);
                return hipGetLastError();
            default:
                break;
        }
    }
    if (C % RPS == 0 && C / RPS <= 16) {
        const dim3 grid(n_chunks, BH);
        switch (C / RPS) {
            case 1:
                hipLaunchKernelGGL((summary_kernel_reg<D, T, 1, RF>), grid, dim3(kSummaryThreads), 0, stream, k, v, ks,
                                   vs, L, n_chunks, eps, rf_scale);
                return hipGetLastError();
            case 2:
                hipLaunchKernelGGL((summary_kernel_reg<D, T, 2, RF>), grid, dim3(kSummaryThreads), 0, stream, k, v, ks,
                                   vs, L, n_chunks, eps, rf_scale);
                return hipGetLastError();
            case 4:
                hipLaunchKernelGGL((summary_kernel_reg<D, T, 4, RF>), grid, dim3(kSummaryThreads), 0, stream, k, v, ks,
                                   vs, L, n_chunks, eps, rf_scale);
                return hipGetLastError();
            case 8:
                hipLaunchKernelGGL((summary_kernel_reg<D, T, 8, RF>), grid, dim3(kSummaryThreads), 0, stream, k, v, ks,
                                   vs, L, n_chunks, eps, rf_scale);
                return hipGetLastError();
            case 16:
                if constexpr (sizeof(T) == 2) {  // bf16 only: 16 rows of fp32 would not fit the registers
                    hipLaunchKernelGGL((summary_kernel_reg<D, T, 16, RF>), grid, dim3(kSummaryThreads), 0, stream, k,
                                       v, ks, vs, L, n_chunks, eps, rf_scale);
                    return hipGetLastError();
                }
                break;
            default:
                break;
        }
    }
    const size_t lds = (size_t)(C + summary_red_floats<D>()) * sizeof(float);
    hipLaunchKernelGGL((summary_kernel<D, T, RF>), dim3(n_chunks, BH), dim3(kSummaryThreads), lds, stream, k, v, ks, vs,
                       L, C, n_chunks, eps, rf_scale);
    return hipGetLastError();
}

}  // namespace

template <int D>
__global__ __launch_bounds__(256) void rf_noise_kernel(float* __restrict__ eps, long long n_blocks,
                                                       int n_chunks, unsigned long long seed) {
    // one thread per block of 4 features: (seq, chunk, i)
    const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_blocks) return;
    const int i = (int)(t % (D / 4));
    const long long sc = t / (D / 4);
    const int chunk = (int)(sc % n_chunks);
    const int seq = (int)(sc / n_chunks);
    float e[4];
    rf_normals4(seed, (uint32_t)i, (uint32_t)chunk, (uint32_t)seq, e);
    *reinterpret_cast<floatx4*>(eps + t * 4) = floatx4{e[0], e[1], e[2], e[3]};
}

template <int D>
hipError_t launch_rf_noise(float* eps, int n_seq, int n_chunks, unsigned long long seed, hipStream_t stream) {
    const long long n_blocks = (long long)n_seq * n_chunks * (D / 4);
    if (n_blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((rf_noise_kernel<D>), dim3((unsigned)((n_blocks + 255) / 256)), dim3(256), 0, stream, eps,
                       n_blocks, n_chunks, seed);
    return hipGetLastError();
}
template hipError_t launch_rf_noise<64>(float*, int, int, unsigned long long, hipStream_t);
template hipError_t launch_rf_noise<128>(float*, int, int, unsigned long long, hipStream_t);

template <int D, typename T>
hipError_t launch_summaries(const void* K, const void* V, void* Ks, void* Vs, int BH, int L, int C,
                            const float* eps, float rf_scale, hipStream_t stream) {
    if (eps) return launch_summaries_impl<D, T, true>(K, V, Ks, Vs, BH, L, C, eps, rf_scale, stream);
    return launch_summaries_impl<D, T, false>(K, V, Ks, Vs, BH, L, C, nullptr, 0.f, stream);
}

#define EVA_SUMMARIES(D, T)                                                                                       \
    template hipError_t launch_summaries<D, T>(const void*, const void*, void*, void*, int, int, int, const float*, \
                                               float, hipStream_t);
EVA_SUMMARIES(64, bf16)
EVA_SUMMARIES(128, bf16)
EVA_SUMMARIES(64, float)
EVA_SUMMARIES(128, float)
#undef EVA_SUMMARIES

}  // namespace eva
