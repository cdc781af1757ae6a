// Chunk-summary kernel for the prefill path: K, V row-major [BH][L][D] ->
// Ks, Vs row-major [BH][L / C][D].  One workgroup per chunk; HBM bound
// (reads every key and value once, writes two rows per chunk).
#include "eva_kernels.hpp"
#include "summary.hpp"

namespace eva {

namespace {

template <int D, typename T>
__global__ __launch_bounds__(kSummaryThreads) void summary_kernel(const T* __restrict__ K, const T* __restrict__ V,
                                                                  T* __restrict__ Ks, T* __restrict__ Vs, int L,
                                                                  int C, int n_chunks) {
    extern __shared__ float smem[];
    constexpr int TPR = D / 8;
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const size_t row0 = bg * (size_t)L + (size_t)chunk * C;
    RowMajorChunk<D, T> src{K + row0 * D, V + row0 * D};
    float kh[8], vh[8];
    chunk_summary<D>(src, C, smem, smem + C, kh, vh);
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

}  // namespace

template <int D, typename T>
hipError_t launch_summaries(const void* K, const void* V, void* Ks, void* Vs, int BH, int L, int C,
                            hipStream_t stream) {
    const int n_chunks = L / C;
    if (n_chunks == 0) return hipSuccess;
    const size_t lds = (size_t)(C + summary_red_floats<D>()) * sizeof(float);
    hipLaunchKernelGGL((summary_kernel<D, T>), dim3(n_chunks, BH), dim3(kSummaryThreads), lds, stream,
                       static_cast<const T*>(K), static_cast<const T*>(V), static_cast<T*>(Ks),
                       static_cast<T*>(Vs), L, C, n_chunks);
    return hipGetLastError();
}

template hipError_t launch_summaries<64, bf16>(const void*, const void*, void*, void*, int, int, int, hipStream_t);
template hipError_t launch_summaries<128, bf16>(const void*, const void*, void*, void*, int, int, int, hipStream_t);
template hipError_t launch_summaries<64, float>(const void*, const void*, void*, void*, int, int, int, hipStream_t);
template hipError_t launch_summaries<128, float>(const void*, const void*, void*, void*, int, int, int, hipStream_t);

}  // namespace eva
