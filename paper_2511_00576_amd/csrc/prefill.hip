// Fused window + summary EVA prefill for gfx950, fp32 (fp32 storage, fp32
// matrix-core products with v_mfma_f32_16x16x4_f32).  The bf16 path is the
// pipelined kernel of prefill_mfma.hip; this kernel has its own tiling and
// masks and serves fp32 callers (it is pinned to 1e-5 by its own tests).
//
// FlashEVA (section "FlashEVA") rewrites EVA as one softmax attention over an
// augmented key set: the exact keys of the query's local window plus one key
// per chunk summary.  The causal form needs a mask of its own (window band for
// exact keys, "chunk lies fully before the window" for summaries); it is never
// materialized here: each 64-key block is classified per wave, and only blocks
// that straddle a boundary evaluate a per-element range test.
//
// Work decomposition: one workgroup = NW waves = one tile of query columns
// that share one key/value head.  A wave owns 32 columns (two 16-column MFMA
// blocks); with G = H / H_kv query heads per kv head the workgroup packs
// Gt = gcd(G, NW) heads x (32 NW / Gt) positions, so every K/V block staged in
// LDS serves all NW waves.  Per block: S^T = K Q^T on the matrix cores (keys
// are MFMA rows, so each lane owns one query column and its softmax
// statistics stay in registers), online softmax in log2 units, O^T += V^T P^T
// with P taken straight from the S^T accumulators.
//
// Staging: K/V blocks go HBM -> LDS with global_load_lds_dwordx4 (no register
// round trip) into a two-stage LDS ring; block j+1 is requested while block j
// is computed, with one barrier per block.  Rows are stored unpadded with an
// XOR swizzle of their 16-B chunks, chosen so that the 16-B K-fragment reads
// and the 4-B V reads hit distinct banks.
#include <type_traits>

#include "eva_device.hpp"
#include "eva_kernels.hpp"

namespace eva {

namespace {

constexpr int kBN = 64;      // keys per block
constexpr int kQW = 32;      // query columns per wave
constexpr int kNS = 2;       // LDS ring stages
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units)

template <int D, int NW>
struct PCfg {
    static constexpr int ROWB = D * 4;          // bytes per row
    static constexpr int CPR = ROWB / 16;       // 16-B chunks per row
    static constexpr int VEC = 4;               // elements per chunk
    static constexpr int BLK = kBN * ROWB;      // bytes per 64-row block
    static constexpr int NI = BLK / 1024 / NW;  // DMA instructions / wave / array
    static_assert(NI >= 1, "block too small for the workgroup");
};

// Chunk swizzles (position = logical chunk ^ swz(row)).  K rows are read as
// 16-B fragments by 16 lanes holding 16 consecutive rows; V rows by 4-B reads,
// 16 lanes on each of 4 rows spaced 4 apart.
template <int CPR>
__device__ __forceinline__ int swz_k(int r) {
    return CPR >= 16 ? (r & 15) : ((r >> 1) & 7);
}
__device__ __forceinline__ int swz_v(int r) { return 4 * ((r >> 2) & 3); }

// One global_load_lds_dwordx4: every lane moves 16 B from base + voff to
// LDS address M0 + 16 * lane.  Inline asm so that the compiler, which cannot
// see the LDS write, leaves the waits to the kernel.
__device__ __forceinline__ void lds_dma16(const void* base, unsigned voff, const void* lds_dst) {
    const unsigned m0 =
        __builtin_amdgcn_readfirstlane((unsigned)(size_t)(__attribute__((address_space(3))) const void*)lds_dst);
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(m0) : "memory");
}

// VAR: window variant (win_lo / win_hi / sum_lo / sum_hi); masks of edge
// blocks are per element for every variant.
template <int D, int NW, int VAR>
__global__ __launch_bounds__(NW * 64) void prefill_kernel(PrefillParams a) {
    typedef PCfg<D, NW> Cfg;
    constexpr int ROWB = Cfg::ROWB, CPR = Cfg::CPR, VEC = Cfg::VEC, BLK = Cfg::BLK, NI = Cfg::NI;
    constexpr int NQF = D / 16;  // Q fragments (4 features each) per 16-column block
    constexpr int NDB = D / 16;  // 16-feature output blocks

    __shared__ __attribute__((aligned(1024))) unsigned char lds[kNS][2][BLK];

    const float* __restrict__ Q = static_cast<const float*>(a.Q);
    float* __restrict__ O = static_cast<float*>(a.O);

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

    // blocks the workgroup stages: summaries [0, s(n_hi)) (non-causal: all),
    // then the window band
    constexpr bool NC = VAR == kWinNonCausal;
    const int s_hi = NC ? a.n_chunks : sum_lo<VAR>(n_hi, W, C);
    const int nsb = (s_hi + kBN - 1) / kBN;
    const int kb0 = win_lo<VAR>(n0, W, C) / kBN;
    const int kb1 = win_hi<VAR>(n_hi, W, L) / kBN;
    const int nb = nsb + (kb1 - kb0 + 1);

    // what this wave needs: prefix summaries c < ws_hi (all columns: c < ws_lo),
    // non-causal suffix summaries c >= wsx_lo (all columns: c >= wsx_hi), and
    // window keys in [wlo_min, whi_max] (all columns: [wlo_max, whi_min])
    const bool w_active = p0 < L;
    const int wp_last = min(p0 + kQW - 1, L - 1);
    const int ws_hi = w_active ? sum_lo<VAR>(wp_last, W, C) : 0;
    const int ws_lo = sum_lo<VAR>(p0, W, C);
    const int wsx_lo = NC ? sum_hi<VAR>(p0, W, C, L) : 0;
    const int wsx_hi = NC ? sum_hi<VAR>(wp_last, W, C, L) : 0;
    const int wlo_min = win_lo<VAR>(p0, W, C), wlo_max = win_lo<VAR>(wp_last, W, C);
    const int whi_min = win_hi<VAR>(p0, W, L), whi_max = win_hi<VAR>(wp_last, W, L);

    const size_t bg = (size_t)b * a.Hkv + kvh;
    const float* Kbg = static_cast<const float*>(a.K) + bg * (size_t)L * D;
    const float* Vbg = static_cast<const float*>(a.V) + bg * (size_t)L * D;
    const float* Ksbg = static_cast<const float*>(a.Ks) + bg * (size_t)a.n_chunks * D;
    const float* Vsbg = static_cast<const float*>(a.Vs) + bg * (size_t)a.n_chunks * D;
    const size_t bh = (size_t)b * a.H + h;

    // per-column facts (column = query position p0 + cb*16 + c16)
    int col_n[2], col_s[2], col_sx[2], col_lo[2], col_span[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        col_n[cb] = p0 + cb * 16 + c16;
        const int n = min(col_n[cb], L - 1);
        col_s[cb] = sum_lo<VAR>(n, W, C);
        col_sx[cb] = NC ? sum_hi<VAR>(n, W, C, L) : a.n_chunks;
        col_lo[cb] = win_lo<VAR>(n, W, C);
        col_span[cb] = win_hi<VAR>(n, W, L) - col_lo[cb];
    }

    // ---- Q fragments (B operand of S^T = K Q^T): contraction feature for
    //      step st = 4f + e is g * (D/4) + st.  Columns past L hold zeros. ----
    floatx4 qf[2][NQF];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        const int n = col_n[cb];
        const float* qrow = Q + (bh * L + (size_t)min(n, L - 1)) * D;
#pragma unroll
        for (int f = 0; f < NQF; ++f) {
            qf[cb][f] = *reinterpret_cast<const floatx4*>(qrow + g * (D / 4) + f * 4);
            if (n >= L) qf[cb][f] = floatx4{};
        }
    }

    // ---- DMA plan: instruction i of this wave fills LDS bytes
    //      [(i*NW + wave) * 1024, +1024) of each array; lane -> (row, chunk) ----
    int dma_row[NI], dma_off[NI], dma_kcol[NI], dma_vcol[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int byte = (i * NW + wave) * 1024 + lane * 16;
        const int r = byte / ROWB;
        const int pos = (byte % ROWB) / 16;
        dma_row[i] = r;
        dma_off[i] = (i * NW + wave) * 1024;
        dma_kcol[i] = (pos ^ swz_k<CPR>(r)) * VEC;  // source chunk landing at LDS chunk pos
        dma_vcol[i] = (pos ^ swz_v(r)) * VEC;
    }
    auto issue = [&](int j) {
        const int st = j % kNS;
        const bool is_sum = j < nsb;
        const int base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        const int limit = is_sum ? a.n_chunks : L;
        const float* kb = (is_sum ? Ksbg : Kbg) + (size_t)base * D;
        const float* vb = (is_sum ? Vsbg : Vbg) + (size_t)base * D;
        // rows past the end repeat the last valid row: finite, and masked out
        // (keys beyond every query, summaries beyond every s(n))
        const int last = limit - 1 - base;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int row = min(dma_row[i], last);
            lds_dma16(kb, (unsigned)((row * D + dma_kcol[i]) * 4), &lds[st][0][dma_off[i]]);
            lds_dma16(vb, (unsigned)((row * D + dma_vcol[i]) * 4), &lds[st][1][dma_off[i]]);
        }
    };

    // ---- per-lane K read offsets (bytes within a stage array): fragment f of
    // key tile kb is row kb*16 + c16, logical chunk g*(D/16) + f; the swizzle
    // of that row depends on c16 only, so kb adds kb*16*ROWB. ----
    int k_off[NQF];
#pragma unroll
    for (int f = 0; f < NQF; ++f) k_off[f] = c16 * ROWB + (((g * (D / 16) + f) ^ swz_k<CPR>(c16)) << 4);

    floatx4 acc[NDB][2];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) acc[db][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    float l_run[2] = {0.f, 0.f};  // per-lane partial softmax denominators
    floatx4 s[4][2];

    issue(0);
    for (int j = 0; j < nb; ++j) {
        // block j landed (the only request in flight); every wave is done with
        // block j-1, whose stage the request for block j+1 refills
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xc070);  // vmcnt(0) lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (j + 1 < nb) issue(j + 1);

        const bool is_sum = j < nsb;
        const int base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        bool needed, full;
        if (is_sum) {
            const int last = base + kBN - 1;
            needed = base < ws_hi || (NC && w_active && last >= wsx_lo && base < a.n_chunks);
            full = last < ws_lo || (NC && base >= wsx_hi && last < a.n_chunks);
        } else {
            needed = w_active && base <= whi_max && base + kBN - 1 >= wlo_min;
            full = base >= wlo_max && base + kBN - 1 <= whi_min;
        }
        if (!needed) continue;
        const unsigned char* ks = lds[j % kNS][0];
        const unsigned char* vs = lds[j % kNS][1];

        // S^T = K Q^T : s[kb][cb] holds keys base + kb*16 + 4g + i
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) s[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int f = 0; f < NQF; ++f) {
            const unsigned char* kp = ks + k_off[f];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const floatx4 ka = *reinterpret_cast<const floatx4*>(kp + kb * 16 * ROWB);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) s[kb][cb] = mfma_f32(ka[e], qf[cb][f][e], s[kb][cb]);
            }
        }

        // mask (boundary blocks only), branch-free per element; element
        // (kb, i) of lane (g, c16) is key base + kb*16 + 4g + i
        if (!full) {
            if (is_sum) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    // summary x = base + 4g + kb*16 + i valid iff x < s(n), or
                    // (non-causal) sum_hi(n) <= x < n_chunks
                    const int lim = col_s[cb] - base - g * 4;
                    const int lim_x = col_sx[cb] - base - g * 4;
                    const int lim_n = a.n_chunks - base - g * 4;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int x = kb * 16 + i;
                            const bool ok = x < lim || (NC && x >= lim_x && x < lim_n);
                            s[kb][cb][i] = ok ? s[kb][cb][i] : -INFINITY;
                        }
                }
            } else {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const int rel = base + g * 4 - col_lo[cb];  // key - win_lo(n) = rel + kb*16 + i
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const unsigned dist = (unsigned)(rel + kb * 16 + i);  // valid iff lo <= key <= hi
                            s[kb][cb][i] = dist <= (unsigned)col_span[cb] ? s[kb][cb][i] : -INFINITY;
                        }
                }
            }
        }

        // online softmax (log2 units), lazy rescaling
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

        // O^T += V^T P^T; element (key kb*16 + 4g + i, feature db*16 + c16),
        // row swizzle depends on g only
        const int vsw = swz_v(g * 4);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = kb * 16 + g * 4 + i;
#pragma unroll
                for (int db = 0; db < NDB; ++db) {
                    const int off = row * ROWB + (((db * 4 + (c16 >> 2)) ^ vsw) << 4) + (c16 & 3) * 4;
                    const float va = *reinterpret_cast<const float*>(vs + off);
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) acc[db][cb] = mfma_f32(va, s[kb][cb][i], acc[db][cb]);
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
        // natural log of the softmax denominator: sum 2^(x - m_run) = lt
        if (a.lse && g == 0) a.lse[bh * L + n] = (m_run[cb] + __builtin_amdgcn_logf(lt)) * kLn2;
        float* orow = O + (bh * L + (size_t)n) * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
            *reinterpret_cast<floatx4*>(orow + db * 16 + g * 4) = acc[db][cb] * inv;
    }
}

}  // namespace

template <int D, int VAR>
void launch_prefill_var(const PrefillParams& p, hipStream_t stream) {
    hipLaunchKernelGGL((prefill_kernel<D, kPrefillWaves, VAR>), dim3(p.n_tiles), dim3(kPrefillWaves * 64), 0, stream,
                       p);
}

template <int D, typename T>
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
    static_assert(std::is_same<T, float>::value, "the fp32 kernel; bf16 runs launch_prefill_mfma");
    switch (p.window) {
        case kWinChunkAligned: launch_prefill_var<D, kWinChunkAligned>(p, stream); break;
        case kWinBlocked: launch_prefill_var<D, kWinBlocked>(p, stream); break;
        case kWinNonCausal: launch_prefill_var<D, kWinNonCausal>(p, stream); break;
        default: launch_prefill_var<D, kWinSliding>(p, stream); break;
    }
    return hipGetLastError();
}

template hipError_t launch_prefill<64, float>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill<128, float>(const PrefillParams&, hipStream_t);

}  // namespace eva
