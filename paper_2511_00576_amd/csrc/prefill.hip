// Fused window + summary EVA prefill for gfx950.
//
// FlashEVA (section "FlashEVA") rewrites EVA as one softmax attention over an
// augmented key set: the exact keys of the query's local window plus one key
// per chunk summary.  The causal form needs a mask of its own (window band for
// exact keys, "chunk lies fully before the window" for summaries); it is never
// materialized here: each 64-key block is classified per wave, and only blocks
// that straddle a boundary evaluate per-element compares.
//
// Work decomposition: one workgroup = 4 waves = one tile of query columns that
// share one key/value head.  A wave owns 32 columns (two 16-column MFMA
// blocks); with G = H / H_kv query heads per kv head the workgroup packs
// Gt = gcd(G, 4) heads x (128 / Gt) positions, so the K/V blocks staged in LDS
// serve every wave.  Per block: S^T = K Q^T on the matrix cores (keys are MFMA
// rows, so every lane owns one query column and its softmax statistics stay in
// registers), online softmax in log2 units, O^T += V^T P^T with P taken
// straight from the S^T accumulators.
//
// Pipeline: the next block's K/V are loaded from HBM into registers while the
// current block is computed from LDS (one LDS stage, register double buffer).
#include "eva_device.hpp"
#include "eva_kernels.hpp"

namespace eva {

namespace {

constexpr int kBN = 64;      // keys per block
constexpr int kQW = 32;      // query columns per wave
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units)

template <int D, typename T>
struct PLayout {
    static constexpr bool BF = sizeof(T) == 2;
    // Row pitches (elements).  bf16: K rows are read 16 B per lane by 8-lane
    // phases -> 272 B pitch (4-bank shift per row); V rows are read by the
    // transposing 8 B read, 4 rows x 32 B per 16-lane group -> 8-bank shift.
    static constexpr int KP = BF ? D + 8 : D + 4;
    static constexpr int VP = BF ? D + 16 : D + 4;
    static constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16-B piece
    static constexpr int PPR = D / VEC;              // pieces per row
    static constexpr int PPT = kBN * PPR / 256;      // pieces per thread
    static constexpr int LDS_BYTES = kBN * (KP + VP) * (int)sizeof(T);
};

template <typename T> struct QFrag;
template <> struct QFrag<bf16> { typedef bf16x8 type; };
template <> struct QFrag<float> { typedef floatx4 type; };

template <int D, typename T>
__global__ __launch_bounds__(256) void prefill_kernel(PrefillParams a) {
    typedef PLayout<D, T> Lay;
    constexpr bool BF = Lay::BF;
    constexpr int NQF = BF ? D / 32 : D / 16;  // Q fragments per 16-column block
    constexpr int NDB = D / 16;                // 16-feature output blocks

    __shared__ __attribute__((aligned(16))) T lds_k[kBN * Lay::KP];
    __shared__ __attribute__((aligned(16))) T lds_v[kBN * Lay::VP];

    const T* __restrict__ Q = static_cast<const T*>(a.Q);
    const T* __restrict__ K = static_cast<const T*>(a.K);
    const T* __restrict__ V = static_cast<const T*>(a.V);
    const T* __restrict__ Ks = static_cast<const T*>(a.Ks);
    const T* __restrict__ Vs = static_cast<const T*>(a.Vs);
    T* __restrict__ O = static_cast<T*>(a.O);

    // ---- tile decode: XCD-aware remap, heavy (late) position tiles first ----
    int id = blockIdx.x;
    {
        const int per = a.n_tiles / 8;
        if (id < per * 8) id = (id % 8) * per + id / 8;
    }
    const int pt = a.n_pos_tiles - 1 - id % a.n_pos_tiles;
    int rest = id / a.n_pos_tiles;
    const int hg = rest % a.n_hg;
    rest /= a.n_hg;
    const int kvh = rest % a.Hkv;
    const int b = rest / a.Hkv;

    const int L = a.L, W = a.W, C = a.C;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, c16 = lane & 15;

    const int h = kvh * a.G + hg * a.Gt + (wave % a.Gt);
    const int n0 = pt * a.pos_per_wg;
    const int p0 = n0 + (wave / a.Gt) * kQW;
    const int n_hi = min(n0 + a.pos_per_wg - 1, L - 1);

    // blocks the workgroup stages: summaries [0, s(n_hi)), then the window band
    const int s_hi = visible_summaries(n_hi, W, C);
    const int nsb = (s_hi + kBN - 1) / kBN;
    const int kb0 = max(0, n0 - W + 1) / kBN;
    const int kb1 = n_hi / kBN;
    const int nb = nsb + (kb1 - kb0 + 1);

    // what this wave needs
    const bool w_active = p0 < L;
    const int wp_last = min(p0 + kQW - 1, L - 1);
    const int ws_hi = w_active ? visible_summaries(wp_last, W, C) : 0;
    const int ws_lo = visible_summaries(p0, W, C);

    const size_t bg = (size_t)b * a.Hkv + kvh;
    const T* Kbg = K + bg * (size_t)L * D;
    const T* Vbg = V + bg * (size_t)L * D;
    const T* Ksbg = Ks + bg * (size_t)a.n_chunks * D;
    const T* Vsbg = Vs + bg * (size_t)a.n_chunks * D;
    const size_t bh = (size_t)b * a.H + h;

    // per-column facts (column = query position p0 + cb*16 + c16)
    int col_n[2], col_s[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        col_n[cb] = p0 + cb * 16 + c16;
        col_s[cb] = visible_summaries(col_n[cb], W, C);
    }

    // ---- Q fragments (B operand of S^T = K Q^T) ----
    typename QFrag<T>::type qf[2][NQF];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        const int n = col_n[cb];
        const T* qrow = Q + (bh * L + (size_t)min(n, L - 1)) * D;
#pragma unroll
        for (int f = 0; f < NQF; ++f) {
            if constexpr (BF) {
                // contraction features dc*32 + 8g .. +7
                qf[cb][f] = *reinterpret_cast<const bf16x8*>(qrow + f * 32 + g * 8);
            } else {
                // contraction feature for step st = 4f+e is g*(D/4) + st
                qf[cb][f] = *reinterpret_cast<const floatx4*>(qrow + g * (D / 4) + f * 4);
            }
            if (n >= L) qf[cb][f] = typename QFrag<T>::type{};
        }
    }

    floatx4 acc[NDB][2];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) acc[db][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    float l_run[2] = {0.f, 0.f};

    // ---- staging: 16-B pieces, thread tid takes pieces tid + 256 i ----
    u32x4 kst[Lay::PPT], vst[Lay::PPT];
    auto load_block = [&](int j) {
        const bool is_sum = j < nsb;
        const int base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        const int limit = is_sum ? a.n_chunks : L;
        const T* kb = is_sum ? Ksbg : Kbg;
        const T* vb = is_sum ? Vsbg : Vbg;
#pragma unroll
        for (int i = 0; i < Lay::PPT; ++i) {
            const int p = tid + 256 * i;
            const int row = base + p / Lay::PPR;
            const int col = (p % Lay::PPR) * Lay::VEC;
            if (row < limit) {
                kst[i] = *reinterpret_cast<const u32x4*>(kb + (size_t)row * D + col);
                vst[i] = *reinterpret_cast<const u32x4*>(vb + (size_t)row * D + col);
            } else {
                kst[i] = u32x4{0u, 0u, 0u, 0u};
                vst[i] = u32x4{0u, 0u, 0u, 0u};
            }
        }
    };
    auto store_block = [&]() {
#pragma unroll
        for (int i = 0; i < Lay::PPT; ++i) {
            const int p = tid + 256 * i;
            const int r = p / Lay::PPR;
            const int col = (p % Lay::PPR) * Lay::VEC;
            *reinterpret_cast<u32x4*>(&lds_k[r * Lay::KP + col]) = kst[i];
            *reinterpret_cast<u32x4*>(&lds_v[r * Lay::VP + col]) = vst[i];
        }
    };

    load_block(0);
    for (int j = 0; j < nb; ++j) {
        __syncthreads();
        store_block();
        __syncthreads();
        if (j + 1 < nb) load_block(j + 1);

        const bool is_sum = j < nsb;
        const int base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        bool needed, full;
        if (is_sum) {
            needed = base < ws_hi;
            full = base + kBN - 1 < ws_lo;
        } else {
            needed = w_active && base <= wp_last && base + kBN - 1 >= p0 - W + 1;
            full = base >= wp_last - W + 1 && base + kBN - 1 <= p0;
        }
        if (!needed) continue;

        // ---- S^T = K Q^T : s[kb][cb] holds keys base + kb*16 + 4g + i ----
        floatx4 s[4][2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) s[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        if constexpr (BF) {
            const T* kl = lds_k + c16 * Lay::KP + g * 8;
#pragma unroll
            for (int dc = 0; dc < D / 32; ++dc) {
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kl + kb * 16 * Lay::KP + dc * 32);
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) s[kb][cb] = mfma_bf16(ka, qf[cb][dc], s[kb][cb]);
                }
            }
        } else {
            const T* kl = lds_k + c16 * Lay::KP + g * (D / 4);
#pragma unroll
            for (int f = 0; f < NQF; ++f) {
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const floatx4 ka = *reinterpret_cast<const floatx4*>(kl + kb * 16 * Lay::KP + f * 4);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int cb = 0; cb < 2; ++cb) s[kb][cb] = mfma_f32(ka[e], qf[cb][f][e], s[kb][cb]);
                }
            }
        }

        // ---- mask (boundary blocks only), branch-free per element ----
        // element (kb, i) of lane (g, c16) is key base + kb*16 + 4g + i
        if (!full) {
            if (is_sum) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const int lim = col_s[cb] - base - g * 4;  // valid iff kb*16 + i < lim
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            s[kb][cb][i] = (kb * 16 + i < lim) ? s[kb][cb][i] : -INFINITY;
                }
            } else {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const int rel = col_n[cb] - base - g * 4;  // n - key = rel - (kb*16 + i)
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const unsigned dist = (unsigned)(rel - (kb * 16 + i));  // valid iff 0 <= n-key < W
                            s[kb][cb][i] = dist < (unsigned)W ? s[kb][cb][i] : -INFINITY;
                        }
                }
            }
        }

        // ---- online softmax (log2 units), lazy rescaling ----
        const float bias = is_sum ? a.log2C : 0.f;
        float bmax[2];
        bool need[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[kb][cb][i]);
            mx = xgroup_max(mx);
            bmax[cb] = mx * a.scale_log2 + bias;  // -inf stays -inf
            need[cb] = bmax[cb] > m_run[cb] + kTau;
        }
        if (__ballot(need[0] || need[1]) != 0) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const float m_new = need[cb] ? bmax[cb] : m_run[cb];
                const float alpha = need[cb] ? fast_exp2(m_run[cb] - m_new) : 1.f;
                l_run[cb] *= alpha;
#pragma unroll
                for (int db = 0; db < NDB; ++db) acc[db][cb] *= alpha;
                m_run[cb] = m_new;
            }
        }
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const float off = bias - (m_run[cb] == -INFINITY ? 0.f : m_run[cb]);
            float ls = 0.f;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p = fast_exp2(fmaf(s[kb][cb][i], a.scale_log2, off));
                    s[kb][cb][i] = p;
                    ls += p;
                }
            l_run[cb] += ls;
        }

        // ---- O^T += V^T P^T ----
        if constexpr (BF) {
            bf16x8 pf[2][2];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        pf[kc][cb][i] = to_bf16(s[2 * kc][cb][i]);
                        pf[kc][cb][4 + i] = to_bf16(s[2 * kc + 1][cb][i]);
                    }
            // transposing read: lane (g, 4j'+t) names V row 4g+j', features 4t..4t+3
            const T* vl = lds_v + (g * 4 + (c16 >> 2)) * Lay::VP + (c16 & 3) * 4;
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const shortx4 lo = lds_read_tr16(vl + (kc * 32) * Lay::VP + db * 16);
                    const shortx4 hi = lds_read_tr16(vl + (kc * 32 + 16) * Lay::VP + db * 16);
                    const bf16x8 va = __builtin_bit_cast(
                        bf16x8, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3],
                                                                              hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) acc[db][cb] = mfma_bf16(va, pf[kc][cb], acc[db][cb]);
                }
            }
        } else {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const T* vr = lds_v + (kb * 16 + g * 4 + i) * Lay::VP + c16;
#pragma unroll
                    for (int db = 0; db < NDB; ++db) {
                        const float va = vr[db * 16];
#pragma unroll
                        for (int cb = 0; cb < 2; ++cb) acc[db][cb] = mfma_f32(va, s[kb][cb][i], acc[db][cb]);
                    }
                }
        }
    }

    // ---- epilogue: O = acc / l ----
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        const float lt = xgroup_sum(l_run[cb]);
        const int n = col_n[cb];
        if (n >= L) continue;
        const float inv = 1.f / lt;
        T* orow = O + (bh * L + (size_t)n) * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const floatx4 v = acc[db][cb] * inv;
            if constexpr (BF) {
                u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *reinterpret_cast<u32x2*>(orow + db * 16 + g * 4) = w;
            } else {
                *reinterpret_cast<floatx4*>(orow + db * 16 + g * 4) = v;
            }
        }
    }
}

}  // namespace

template <int D, typename T>
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
    hipLaunchKernelGGL((prefill_kernel<D, T>), dim3(p.n_tiles), dim3(256), 0, stream, p);
    return hipGetLastError();
}

template hipError_t launch_prefill<64, bf16>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill<128, bf16>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill<64, float>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill<128, float>(const PrefillParams&, hipStream_t);

}  // namespace eva
