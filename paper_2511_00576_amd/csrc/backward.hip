// Backward pass of the fused EVA prefill (bf16, every window variant): dQ, dK, dV
// of a loss given dO, through the window keys/values, the summary keys and
// values, and the summaries' own dependence on K and V.
//
// Notation: logits l = q.k / sqrt(d) (+ ln C for a summary), the row's
// softmax P = exp(l - lse) with lse saved by the forward, D = dO . O per row,
// dS = P (dP - D) with dP = dO . v.  Then dq = sum dS k / sqrt(d),
// dk += dS q / sqrt(d), dv += P dO (FlashAttention-style recomputation: no
// attention matrix is stored).
//
// Kernels (all bf16 storage, fp32 arithmetic, v_mfma_f32_16x16x32_bf16):
//   bwd_dq_kernel      per query tile (4 waves x 16 columns of one head): the
//                      columns' D = dO . O (stored for the dK/dV kernels), then key
//                      blocks of 32 rows (summaries then window band) streamed
//                      through LDS: S^T = K Q^T, dP^T = V dO^T, dS^T, and
//                      dQ^T += K^T dS^T (K^T by the transposing LDS read)
//   bwd_dkdv_kernel    per key tile (4 waves x 16 keys, window keys or
//                      summaries of one kv head), query blocks of 32 rows of
//                      every head of the group streamed through LDS:
//                      S = Q K^T, dP = dO V^T, dS, dV^T += dO^T P,
//                      dK^T += Q^T dS.  Summary tiles run first and leave
//                      fp32 summary gradients; window tiles run last and add
//                      each key's share of its chunk's summary gradient
//                      before storing dK, dV as bf16
//   bwd_summary_kernel per chunk, between the two: through khat = mean and
//                      the chunk softmax (vhat = sum_j b_j v_j,
//                      b = softmax(khat . k / sqrt(d))); leaves khat, the
//                      total gradient of khat, and each key's b_j and
//                      logit gradient da_j, from which
//                        dk_j += da_j khat / sqrt(d) + dkhat / C,
//                        dv_j += b_j dvhat
// The fragment layouts are those of the forward kernel: streamed rows are the
// A operand (16-B row reads, or transposing reads for the transposed
// products), the stationary rows are B-operand fragments in registers, and
// the 16x16 score tiles of two key (or query) halves form the next product's
// B operand in place.
#include <type_traits>

#include "eva_device.hpp"
#include "eva_kernels.hpp"
#include "summary.hpp"

namespace eva {

namespace {

constexpr int kBwdWaves = 4;
constexpr int kBwdBN = 32;     // rows per streamed block
// dQ: 16 query columns per wave (122 VGPRs), a two-stage ring (33 KB): four
// workgroups per CU.  Measured on MI355X: the dQ kernel 588 us against 640
// with three stages at three workgroups per CU (LLM and GQA workloads
// averaged); earlier, 537 us (LLM) with three stages vs 568 with 32 columns
// at two waves per SIMD and 634 with 32 columns and four stages.
constexpr int kDqColBlocks = 1, kDqNS = 2, kDqWpe = 4;
// dK/dV: LDS ring stages and blocks requested ahead of the one computed.
// It fits 168 VGPRs, so three stages (50 KB) let three workgroups share a CU
// (measured on MI355X: 631 vs 767 us for the window tiles of the LLM workload)
constexpr int kKvNS = 3, kKvAhead = 2;

// s_waitcnt vmcnt(N) lgkmcnt(0): the kernel's own DMA requests are invisible
// to the compiler, so every wait for them is explicit
template <int N>
__device__ __forceinline__ void bwait_vm() {
    static_assert(N < 64, "vmcnt field is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}
// wait for a block (LATER DMA instructions issued after it may stay in
// flight), then a workgroup barrier: the block is visible to every wave, and
// every wave is done with the stage the next request refills
template <int LATER>
__device__ __forceinline__ void bsync() {
    asm volatile("" ::: "memory");
    bwait_vm<LATER>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int D>
struct BCfg {
    static constexpr int ROWB = 2 * D;            // bytes per row
    static constexpr int CPR = ROWB / 16;         // 16-B chunks per row
    static constexpr int BLK = kBwdBN * ROWB;     // bytes per block
    static constexpr int NI = BLK / 1024 / kBwdWaves;  // DMA instructions per wave per array
    static constexpr int NDC = D / 32;            // contraction steps over features
    static constexpr int NDB = D / 16;            // 16-feature output blocks
};

// stored 16-B chunk = logical chunk ^ bswz(row): conflict-free 16-B row reads
template <int CPR>
__device__ __forceinline__ int bswz(int r) {
    return CPR >= 16 ? (r & 15) : ((r >> 1) & 7);
}

__device__ __forceinline__ void bdma16(const void* base, unsigned voff, unsigned lds_addr) {
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

template <int D>
struct Stager {
    typedef BCfg<D> Cfg;
    int row[Cfg::NI], off[Cfg::NI];  // per DMA instruction: source row and chunk byte offset
    __device__ Stager(int wave, int lane) {
#pragma unroll
        for (int i = 0; i < Cfg::NI; ++i) {
            const int byte = (i * kBwdWaves + wave) * 1024 + lane * 16;
            const int r = byte / Cfg::ROWB;
            const int pos = (byte % Cfg::ROWB) / 16;
            row[i] = r;
            off[i] = (pos ^ bswz<Cfg::CPR>(r)) << 4;
        }
    }
    // rows [0, n_valid) of `src` (row-major, D bf16 each) into the LDS block at
    // lds_addr; rows past n_valid repeat the last valid row (finite, masked).
    // With real false the same number of instructions read row 0 of src into
    // the 1-KB area at lds_addr (requests past the last block).
    __device__ void issue(const bf16* src, int n_valid, unsigned lds_addr, int wave, bool real = true) const {
#pragma unroll
        for (int i = 0; i < Cfg::NI; ++i) {
            const int r = real ? min(row[i], n_valid - 1) : 0;
            bdma16(src, (unsigned)(r * Cfg::ROWB + off[i]), real ? lds_addr + (i * kBwdWaves + wave) * 1024 : lds_addr);
        }
    }
};

template <int D>
__device__ __forceinline__ unsigned lds_addr_of(const void* p) {
    return (unsigned)(size_t)(__attribute__((address_space(3))) const void*)p;
}

// 16-B row fragment: row kb*16 + c16, features dc*32 + 8g .. +7
template <int D>
__device__ __forceinline__ bf16x8 row_frag(const unsigned char* blk, int kb, int dc, int c16, int g) {
    typedef BCfg<D> Cfg;
    const int r = kb * 16 + c16;
    const int chunk = (dc * 4 + g) ^ bswz<Cfg::CPR>(r);
    return *reinterpret_cast<const bf16x8*>(blk + r * Cfg::ROWB + chunk * 16);
}

// transposing fragment (A operand of a transposed product): lane (g, c16)
// receives feature db*16 + c16 of rows 4g .. 4g+3 and 16+4g .. 16+4g+3
template <int D>
__device__ __forceinline__ bf16x8 tr_frag(const unsigned char* blk, int db, int c16, int g) {
    typedef BCfg<D> Cfg;
    const int r = g * 4 + (c16 >> 2);
    const int t = c16 & 3;
    const int chunk = (2 * db + (t >> 1)) ^ bswz<Cfg::CPR>(r);
    const unsigned char* p = blk + r * Cfg::ROWB + chunk * 16 + (t & 1) * 8;
    const shortx4 lo = lds_read_tr16(reinterpret_cast<const bf16*>(p));
    // row r + 16 has the same swizzle (bswz depends on r mod 16)
    const shortx4 hi = lds_read_tr16(reinterpret_cast<const bf16*>(p + 16 * Cfg::ROWB));
    return __builtin_bit_cast(
        bf16x8, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
}

// B-operand fragment in the contraction order of tr_frag: element e is tile
// kb = e / 4, row 4g + e % 4 of a pair of 16x16 output tiles
__device__ __forceinline__ bf16x8 pair_to_b(const floatx4& t0, const floatx4& t1) {
    bf16x8 f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[i] = to_bf16(t0[i]);
        f[4 + i] = to_bf16(t1[i]);
    }
    return f;
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
template <int D, int NCB, int NS, int WPE, int VAR>
__global__ __launch_bounds__(kBwdWaves * 64) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void bwd_dq_kernel(BwdParams a) {
    typedef BCfg<D> Cfg;
    constexpr int NDC = Cfg::NDC, NDB = Cfg::NDB, BLK = Cfg::BLK;
    constexpr int CW = 16 * NCB;       // query columns per wave
    constexpr int AHEAD = NS - 1;      // blocks requested ahead of the one computed
    static_assert(NS == 2 || NS == 3, "the block loop below takes NS steps per trip");
    __shared__ __attribute__((aligned(1024))) unsigned char lds[NS][2][BLK];  // [stage][K, V]
    __shared__ __attribute__((aligned(1024))) unsigned char dummy[1024];

    const int L = a.L, W = a.W, C = a.C;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    constexpr int POS = kBwdWaves * CW;  // positions per workgroup
    const int n_pt = (L + POS - 1) / POS;
    const int pt = n_pt - 1 - (int)blockIdx.x % n_pt;  // late (heavy) tiles first
    const int bh = (int)blockIdx.x / n_pt;
    const int b = bh / a.H, h = bh % a.H;
    const int kvh = h / (a.H / a.Hkv);
    const size_t bg = (size_t)b * a.Hkv + kvh;
    const int n0 = pt * POS;
    const int n_hi = min(n0 + POS - 1, L - 1);
    const int p0 = n0 + wave * CW;
    const bool w_active = p0 < L;
    const int wp_last = min(p0 + CW - 1, L - 1);

    // block plan as in the forward: summaries [0, sum_lo(n_hi)) (non-causal:
    // all), then the window band [win_lo(n0), win_hi(n_hi)]
    constexpr bool NC = VAR == kWinNonCausal;
    const int nsb = ((NC ? a.n_chunks : sum_lo<VAR>(n_hi, W, C)) + kBwdBN - 1) / kBwdBN;
    const int kb0 = win_lo<VAR>(n0, W, C) / kBwdBN;
    const int nb = nsb + (win_hi<VAR>(n_hi, W, L) / kBwdBN - kb0 + 1);
    // what this wave needs: prefix summaries c < ws_hi (all columns: c < ws_lo),
    // non-causal suffix summaries c >= wsx_lo (all columns: c >= wsx_hi), and
    // window keys in [wlo_min, whi_max] (all columns: [wlo_max, whi_min])
    const int ws_hi = w_active ? sum_lo<VAR>(wp_last, W, C) : 0;
    const int ws_lo = sum_lo<VAR>(p0, W, C);
    const int wsx_lo = NC ? sum_hi<VAR>(p0, W, C, L) : 0;
    const int wsx_hi = NC ? sum_hi<VAR>(wp_last, W, C, L) : 0;
    const int wlo_min = win_lo<VAR>(p0, W, C), wlo_max = win_lo<VAR>(wp_last, W, C);
    const int whi_min = win_hi<VAR>(p0, W, L), whi_max = win_hi<VAR>(wp_last, W, L);

    const bf16* Kbg = static_cast<const bf16*>(a.K) + bg * (size_t)L * D;
    const bf16* Vbg = static_cast<const bf16*>(a.V) + bg * (size_t)L * D;
    const bf16* Ksbg = static_cast<const bf16*>(a.Ks) + bg * (size_t)a.n_chunks * D;
    const bf16* Vsbg = static_cast<const bf16*>(a.Vs) + bg * (size_t)a.n_chunks * D;

    // stationary columns: q and dO fragments (B operands), lse and D
    const size_t row0 = (size_t)bh * L;
    bf16x8 qf[NCB][NDC], gf[NCB][NDC];
    float lse2[NCB], dcol[NCB];
    int col_n[NCB], col_s[NCB], col_sx[NCB], col_lo[NCB], col_span[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        col_n[cb] = p0 + cb * 16 + c16;
        const int n = min(col_n[cb], L - 1);
        col_s[cb] = sum_lo<VAR>(n, W, C);
        col_sx[cb] = NC ? sum_hi<VAR>(n, W, C, L) : a.n_chunks;
        col_lo[cb] = win_lo<VAR>(n, W, C);
        col_span[cb] = win_hi<VAR>(n, W, L) - col_lo[cb];
        const bf16* qrow = static_cast<const bf16*>(a.Q) + (row0 + n) * D;
        const bf16* grow = static_cast<const bf16*>(a.dO) + (row0 + n) * D;
        const bf16* orow = static_cast<const bf16*>(a.O) + (row0 + n) * D;
        const bf16* lrow = a.O_lo ? static_cast<const bf16*>(a.O_lo) + (row0 + n) * D : nullptr;
        // D = dO . O of the column (O + O_lo when the forward kept its output's
        // rounding residual): this lane's 8 NDC features, then the four lanes
        // (g) of the column; stored for the dK/dV kernels
        float dot = 0.f;
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc) {
            qf[cb][dc] = *reinterpret_cast<const bf16x8*>(qrow + dc * 32 + g * 8);
            gf[cb][dc] = *reinterpret_cast<const bf16x8*>(grow + dc * 32 + g * 8);
            const bf16x8 of = *reinterpret_cast<const bf16x8*>(orow + dc * 32 + g * 8);
            bf16x8 lf = {};
            if (lrow) lf = *reinterpret_cast<const bf16x8*>(lrow + dc * 32 + g * 8);
#pragma unroll
            for (int e = 0; e < 8; ++e) dot += (float)gf[cb][dc][e] * ((float)of[e] + (float)lf[e]);
        }
        dcol[cb] = xgroup_sum(dot);
        if (g == 0 && col_n[cb] < L) a.Dv[row0 + n] = dcol[cb];
        lse2[cb] = a.lse[row0 + n] * kLog2e;
    }

    floatx4 acc[NDB][NCB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[db][cb] = floatx4{0.f, 0.f, 0.f, 0.f};

    // block j of the plan into stage j % NS; past the last block the same
    // number of DMA instructions go to the dummy area
    const Stager<D> st(wave, lane);
    constexpr int REQ = 2 * Cfg::NI;  // DMA instructions per request and wave
    auto stage = [&](int j) {
        const bool real = j < nb;
        const bool sum = j < nsb;
        const int base = sum ? j * kBwdBN : (kb0 + j - nsb) * kBwdBN;
        const int lim = sum ? a.n_chunks : L;
        const int nv = min(kBwdBN, lim - base);
        const bf16* ksrc = real ? (sum ? Ksbg : Kbg) + (size_t)base * D : Kbg;
        const bf16* vsrc = real ? (sum ? Vsbg : Vbg) + (size_t)base * D : Vbg;
        st.issue(ksrc, nv, lds_addr_of<D>(real ? lds[j % NS][0] : dummy), wave, real);
        st.issue(vsrc, nv, lds_addr_of<D>(real ? lds[j % NS][1] : dummy), wave, real);
    };
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) stage(k);
    // the stationary fragments (plain loads) and the first blocks: the
    // compiler does not count the DMA requests, so its own wait for the
    // fragments would otherwise sit inside the loop and drain every request
    bwait_vm<0>();
    auto block_step = [&](auto ph_tag, int j) {
        constexpr int PH = decltype(ph_tag)::value;  // j mod NS: the stage as a constant
        // block j landed (the AHEAD - 1 requested after it may be in flight);
        // the request below refills the stage of block j-1
        bsync<(AHEAD - 1) * REQ>();
        stage(j + AHEAD);
        const bool sum = j < nsb;
        const int base = sum ? j * kBwdBN : (kb0 + j - nsb) * kBwdBN;
        const int last = base + kBwdBN - 1;
        const bool needed =
            w_active && (sum ? base < ws_hi || (NC && last >= wsx_lo && base < a.n_chunks)
                             : base <= whi_max && last >= wlo_min);
        if (!needed) return;
        const unsigned char* ks = lds[PH][0];
        const unsigned char* vs = lds[PH][1];
        // S^T and dP^T: rows = keys base + kb*16 + 4g + i, column = query c16
        floatx4 s[2][NCB], dp[2][NCB];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) s[kb][cb] = dp[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8 kf = row_frag<D>(ks, kb, dc, c16, g);
                const bf16x8 vf = row_frag<D>(vs, kb, dc, c16, g);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    s[kb][cb] = mfma_bf16(kf, qf[cb][dc], s[kb][cb]);
                    dp[kb][cb] = mfma_bf16(vf, gf[cb][dc], dp[kb][cb]);
                }
            }
        // P^T and dS^T (masked entries: 0); a block every pair of which is
        // visible to this wave's columns skips the per-element test
        const float bias = sum ? a.log2C : 0.f;
        const bool full = wp_last == p0 + CW - 1 &&
                          (sum ? last < ws_lo || (NC && base >= wsx_hi && last < a.n_chunks)
                               : base >= wlo_max && last <= whi_min);
        if (full) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float p = fast_exp2(fmaf(s[kb][cb][i], a.scale_log2, bias - lse2[cb]));
                        s[kb][cb][i] = p * (dp[kb][cb][i] - dcol[cb]);  // dS^T
                    }
        } else {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int n = col_n[cb];
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = base + kb * 16 + g * 4 + i;
                        const bool ok = n < L && (sum ? key < col_s[cb] || (NC && key >= col_sx[cb] &&
                                                                            key < a.n_chunks)
                                                      : (unsigned)(key - col_lo[cb]) <= (unsigned)col_span[cb]);
                        const float p = ok ? fast_exp2(fmaf(s[kb][cb][i], a.scale_log2, bias - lse2[cb])) : 0.f;
                        s[kb][cb][i] = p * (dp[kb][cb][i] - dcol[cb]);  // dS^T
                    }
            }
        }
        bf16x8 dsf[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) dsf[cb] = pair_to_b(s[0][cb], s[1][cb]);
        // dQ^T += K^T dS^T
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const bf16x8 kt = tr_frag<D>(ks, db, c16, g);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) acc[db][cb] = mfma_bf16(kt, dsf[cb], acc[db][cb]);
        }
    };
    // three steps per trip, so that each one's stage index is a constant
    typedef std::integral_constant<int, 0> P0;
    typedef std::integral_constant<int, 1> P1;
    typedef std::integral_constant<int, 2> P2;
    int j = 0;
    if constexpr (NS == 3) {
        for (; j + 2 < nb; j += 3) {
            block_step(P0{}, j);
            block_step(P1{}, j + 1);
            block_step(P2{}, j + 2);
        }
        if (j < nb) block_step(P0{}, j);
        if (j + 1 < nb) block_step(P1{}, j + 1);
    } else {
        for (; j + 1 < nb; j += 2) {
            block_step(P0{}, j);
            block_step(P1{}, j + 1);
        }
        if (j < nb) block_step(P0{}, j);
    }

    bwait_vm<0>();  // no request may still be writing LDS when the workgroup ends

    // dQ = acc / sqrt(d): lane (g, c16) holds features db*16 + 4g .. +3 of column c16
    const float inv_sqrt_d = a.scale_log2 / kLog2e;
    bf16* dQ = static_cast<bf16*>(a.dQ);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const int n = col_n[cb];
        if (n >= L) continue;
        bf16* orow = dQ + (row0 + n) * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const floatx4 v = acc[db][cb] * inv_sqrt_d;
            u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
            *reinterpret_cast<u32x2*>(orow + db * 16 + g * 4) = w;
        }
    }
}

// ---------------------------------------------------------------------------
// dK, dV of window keys and of summaries
// ---------------------------------------------------------------------------
// Rows that see window key m: [kv_rows_lo(m), kv_rows_hi(m)] (the inverse
// of [win_lo(n), win_hi(n)], both non-decreasing); rows that see summary c
// from the prefix side: n >= sum_rows_lo(c) (win_lo(n) >= (c + 1) C).
// Non-causal summaries are also seen by the rows of the blocks wholly before
// them: their tiles stream every row, masked per element.
template <int VAR>
__device__ __forceinline__ int kv_rows_lo(int m, int W) {
    return VAR == kWinNonCausal ? (m / W) * W : m;
}
template <int VAR>
__device__ __forceinline__ long long kv_rows_hi(int m, int W, int C) {
    if constexpr (VAR == kWinSliding) return (long long)m + W - 1;
    if constexpr (VAR == kWinChunkAligned) return ((long long)(m / C) + 1) * C + W - 2;
    return (long long)(m / W) * W + W - 1;
}
template <int VAR>
__device__ __forceinline__ long long sum_rows_lo(int c, int W, int C) {
    if constexpr (VAR == kWinSliding || VAR == kWinChunkAligned) return ((long long)c + 1) * C + W - 1;
    if constexpr (VAR == kWinBlocked) return (((long long)c + 1) * C + W - 1) / W * W;
    return 0;
}

template <int D, bool SUM, int VAR>
__global__ __launch_bounds__(kBwdWaves * 64) __attribute__((amdgpu_waves_per_eu(3, 3))) void bwd_dkdv_kernel(BwdParams a) {
    typedef BCfg<D> Cfg;
    constexpr int NDC = Cfg::NDC, NDB = Cfg::NDB, BLK = Cfg::BLK;
    constexpr int KT = kBwdWaves * 16;  // keys per workgroup
    __shared__ __attribute__((aligned(1024))) unsigned char lds[kKvNS][2][BLK];  // [stage][Q, dO]
    __shared__ __attribute__((aligned(256))) float rowf[kKvNS][2][64];            // [stage][lse, D] of its rows
    __shared__ __attribute__((aligned(1024))) unsigned char dummy[1024];

    const int L = a.L, W = a.W, C = a.C;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    // key tiles per (b, kv head): summaries, or window keys
    constexpr bool sum = SUM;
    // summary tiles: n_split workgroups per tile, each over a part of the
    // query range, leaving partial sums
    const int n_split = SUM ? a.n_split : 1;
    const int per_bg = (SUM ? (a.n_chunks + KT - 1) / KT : (L + KT - 1) / KT) * n_split;
    const int bgi = (int)blockIdx.x / per_bg;
    const int t = (int)blockIdx.x % per_bg / n_split;
    const int sp = (int)blockIdx.x % n_split;
    const size_t bg = (size_t)bgi;
    const int b = bgi / a.Hkv, kvh = bgi % a.Hkv;
    const int G = a.H / a.Hkv;
    const int k0 = t * KT;                        // first key (or summary) of the tile
    const int lim = sum ? a.n_chunks : L;
    const int key = k0 + wave * 16 + c16;         // this lane's key column
    const int key_c = min(key, lim - 1);

    // stationary key/value rows (B operands): features dc*32 + 8g .. +7 of key_c
    const bf16* Kr = static_cast<const bf16*>(sum ? a.Ks : a.K) + (bg * (size_t)lim + key_c) * D;
    const bf16* Vr = static_cast<const bf16*>(sum ? a.Vs : a.V) + (bg * (size_t)lim + key_c) * D;
    bf16x8 kf[NDC], vf[NDC];
#pragma unroll
    for (int dc = 0; dc < NDC; ++dc) {
        kf[dc] = *reinterpret_cast<const bf16x8*>(Kr + dc * 32 + g * 8);
        vf[dc] = *reinterpret_cast<const bf16x8*>(Vr + dc * 32 + g * 8);
    }

    // query rows that can see some key of the tile (and of this wave's keys
    // [wk0, wk1]): window key k is seen by rows [kv_rows_lo(k), kv_rows_hi(k)],
    // summary c by rows from sum_rows_lo(c) on (non-causal: by any row)
    constexpr bool NC = VAR == kWinNonCausal;
    const int k_last = min(k0 + KT, lim) - 1;
    const int r_lo = sum ? (int)min((long long)L, sum_rows_lo<VAR>(k0, W, C)) : kv_rows_lo<VAR>(k0, W);
    const int r_hi = sum ? L - 1 : (int)min((long long)L - 1, kv_rows_hi<VAR>(k_last, W, C));
    const int qb0 = r_lo / kBwdBN;
    const int nqb = r_lo <= r_hi ? r_hi / kBwdBN - qb0 + 1 : 0;
    const int wk0 = k0 + wave * 16, wk1 = min(wk0 + 15, lim - 1);
    const bool w_active = wk0 < lim;
    const int wr_lo = sum ? (int)min((long long)L, sum_rows_lo<VAR>(wk0, W, C)) : kv_rows_lo<VAR>(wk0, W);
    const int wr_hi = sum ? L - 1 : (int)min((long long)L - 1, kv_rows_hi<VAR>(wk1, W, C));

    floatx4 dk[NDB], dv[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db) dk[db] = dv[db] = floatx4{0.f, 0.f, 0.f, 0.f};
    const float bias = sum ? a.log2C : 0.f;

    const Stager<D> stg(wave, lane);
    // (head, query block) pairs [j0, j0 + steps) of the nqb * G the tile sees
    const int all_steps = nqb * G;
    const int j0 = (int)((long long)all_steps * sp / n_split);
    const int steps = (int)((long long)all_steps * (sp + 1) / n_split) - j0;
    // request of step j: its Q and dO rows (stage j % NS), and their lse and D
    // (one 4-B DMA instruction each, by waves 0 and 1; waves 2 and 3 issue one
    // into the dummy area so that every wave counts the same instructions)
    constexpr int REQ = 2 * Cfg::NI + 1;
    static_assert(kKvNS == 3, "the step loop below takes three steps per trip");
    auto stage = [&](int j) {
        const bool real = j < steps;
        // past the last step: row 0 of the group's first head (always valid)
        const int hh = real ? (j0 + j) / nqb : 0, qb = real ? qb0 + (j0 + j) % nqb : 0;
        const size_t rowh = ((size_t)b * a.H + kvh * G + hh) * L;
        const size_t rowb = rowh + (size_t)qb * kBwdBN;
        const int nv = min(kBwdBN, L - qb * kBwdBN);
        const int st_i = j % kKvNS;
        stg.issue(static_cast<const bf16*>(a.Q) + rowb * D, nv, lds_addr_of<D>(real ? lds[st_i][0] : dummy), wave, real);
        stg.issue(static_cast<const bf16*>(a.dO) + rowb * D, nv, lds_addr_of<D>(real ? lds[st_i][1] : dummy), wave,
                  real);
        const bool mine = real && wave < 2;
        const float* src = wave == 1 ? a.Dv : a.lse;
        const unsigned voff = (unsigned)(mine ? min(lane, nv - 1) : 0) * 4u;
        const unsigned dst = mine ? lds_addr_of<D>(rowf[st_i][wave]) : lds_addr_of<D>(dummy);
        asm volatile("global_load_lds_dword %0, %1" ::"v"(voff), "s"(src + rowb),
                     "{m0}"(__builtin_amdgcn_readfirstlane(dst))
                     : "memory");
    };
#pragma unroll
    for (int k = 0; k < kKvAhead; ++k) stage(k);
    // see bwd_dq_kernel: the stationary fragments are waited for here
    bwait_vm<0>();
    auto block_step = [&](auto ph_tag, int j) {
        constexpr int PH = decltype(ph_tag)::value;  // j mod NS: the stage as a constant
        // step j's rows landed (the request after it may be in flight); the
        // request below refills the stage of step j-1
        bsync<(kKvAhead - 1) * REQ>();
        stage(j + kKvAhead);
        const int qb = qb0 + (j0 + j) % nqb;
        const int r0 = qb * kBwdBN;
        if (!w_active || r0 > wr_hi || r0 + kBwdBN - 1 < wr_lo) return;
        constexpr int st_i = PH;
        // lse and D of this lane's 8 query rows r0 + 16 kb + 4g + i
        float lse2[2][4], dq[2][4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const floatx4 l4 = *reinterpret_cast<const floatx4*>(&rowf[st_i][0][kb * 16 + g * 4]);
            const floatx4 d4 = *reinterpret_cast<const floatx4*>(&rowf[st_i][1][kb * 16 + g * 4]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                lse2[kb][i] = l4[i] * kLog2e;
                dq[kb][i] = d4[i];
            }
        }
        const unsigned char* qs = lds[st_i][0];
        const unsigned char* gs = lds[st_i][1];
        // S and dP: rows = queries r0 + kb*16 + 4g + i, column = key c16
        floatx4 s[2], dp[2];
        s[0] = s[1] = dp[0] = dp[1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                s[kb] = mfma_bf16(row_frag<D>(qs, kb, dc, c16, g), kf[dc], s[kb]);
                dp[kb] = mfma_bf16(row_frag<D>(gs, kb, dc, c16, g), vf[dc], dp[kb]);
            }
        floatx4 p[2];
        // a step every pair of which is visible (the wave's 16 keys, the
        // block's 32 rows: most window steps) skips the per-element test
        const int r1 = r0 + kBwdBN - 1;
        const bool full = wk0 + 15 < lim && r1 < L &&
                          (sum ? wk0 + 16 <= sum_lo<VAR>(r0, W, C) ||
                                     (NC && wk0 >= sum_hi<VAR>(r1, W, C, L))
                               : win_lo<VAR>(r1, W, C) <= wk0 && wk0 + 15 <= win_hi<VAR>(r0, W, L));
        if (full) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    p[kb][i] = fast_exp2(fmaf(s[kb][i], a.scale_log2, bias - lse2[kb][i]));
                    s[kb][i] = p[kb][i] * (dp[kb][i] - dq[kb][i]);  // dS
                }
        } else {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = r0 + kb * 16 + g * 4 + i;
                    const int nc = min(n, L - 1);
                    const bool ok = key < lim && n < L &&
                                    (sum ? key < sum_lo<VAR>(nc, W, C) || (NC && key >= sum_hi<VAR>(nc, W, C, L))
                                         : win_lo<VAR>(nc, W, C) <= key && key <= win_hi<VAR>(nc, W, L));
                    p[kb][i] = ok ? fast_exp2(fmaf(s[kb][i], a.scale_log2, bias - lse2[kb][i])) : 0.f;
                    s[kb][i] = p[kb][i] * (dp[kb][i] - dq[kb][i]);  // dS
                }
        }
        const bf16x8 pf = pair_to_b(p[0], p[1]);
        const bf16x8 dsf = pair_to_b(s[0], s[1]);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            dv[db] = mfma_bf16(tr_frag<D>(gs, db, c16, g), pf, dv[db]);
            dk[db] = mfma_bf16(tr_frag<D>(qs, db, c16, g), dsf, dk[db]);
        }
    };
    // three steps per trip, so that each one's stage index is a constant
    typedef std::integral_constant<int, 0> P0;
    typedef std::integral_constant<int, 1> P1;
    typedef std::integral_constant<int, 2> P2;
    int j = 0;
    for (; j + 2 < steps; j += 3) {
        block_step(P0{}, j);
        block_step(P1{}, j + 1);
        block_step(P2{}, j + 2);
    }
    if (j < steps) block_step(P0{}, j);
    if (j + 1 < steps) block_step(P1{}, j + 1);

    bwait_vm<0>();  // no request may still be writing LDS when the workgroup ends
    if (key >= lim) return;
    const float inv_sqrt_d = a.scale_log2 / kLog2e;
    if constexpr (SUM) {
        // fp32 partial summary gradients, for the per-chunk pass
        const size_t slot = (size_t)sp * a.B * a.Hkv * lim;
        float* dKo = a.dKs_w + (slot + bg * (size_t)lim + key) * D;
        float* dVo = a.dVs_w + (slot + bg * (size_t)lim + key) * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            *reinterpret_cast<floatx4*>(dKo + db * 16 + g * 4) = dk[db] * inv_sqrt_d;
            *reinterpret_cast<floatx4*>(dVo + db * 16 + g * 4) = dv[db];
        }
    } else {
        // window gradient plus the key's share of its chunk's summary gradient
        // (keys after the last complete chunk have none)
        const int c = key / C;
        const bool in_chunk = c < a.n_chunks;
        float da = 0.f, bj = 0.f;
        const size_t cv = (bg * (size_t)a.n_chunks + (in_chunk ? c : 0)) * D;
        if (in_chunk) {
            da = a.da_w[bg * (size_t)a.n_chunks * C + key] * inv_sqrt_d;
            bj = a.bw_w[bg * (size_t)a.n_chunks * C + key];
        }
        bf16* dKo = static_cast<bf16*>(a.dK) + (bg * (size_t)L + key) * D;
        bf16* dVo = static_cast<bf16*>(a.dV) + (bg * (size_t)L + key) * D;
        const float inv_c = 1.f / (float)C;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            floatx4 gk = dk[db] * inv_sqrt_d, gv = dv[db];
            if (in_chunk) {
                const int f = db * 16 + g * 4;
                const floatx4 kh = *reinterpret_cast<const floatx4*>(a.khat_w + cv + f);
                const floatx4 dkh = *reinterpret_cast<const floatx4*>(a.dkhat_w + cv + f);
                const floatx4 dvh = *reinterpret_cast<const floatx4*>(a.dVs_w + cv + f);
                gk += da * kh + dkh * inv_c;
                gv += bj * dvh;
            }
            const u32x2 wk = {pack_bf16x2(gk[0], gk[1]), pack_bf16x2(gk[2], gk[3])};
            const u32x2 wv = {pack_bf16x2(gv[0], gv[1]), pack_bf16x2(gv[2], gv[3])};
            *reinterpret_cast<u32x2*>(dKo + db * 16 + g * 4) = wk;
            *reinterpret_cast<u32x2*>(dVo + db * 16 + g * 4) = wv;
        }
    }
}

// ---------------------------------------------------------------------------
// through the summaries, plus the window gradients, to dK and dV
// ---------------------------------------------------------------------------
// One 256-thread workgroup per chunk.  Thread t holds features cc*8 ..
// cc*8+7 (cc = t % TPR) of rows r0, r0 + RPS, ... (r0 = t / TPR).  LDS: a_j
// (log2 units), C floats, the reduction scratch, then the chunk's summary
// gradients (2 D floats).
template <int D>
__global__ __launch_bounds__(256) void bwd_summary_kernel(BwdParams a) {
    constexpr int TPR = D / 8;
    constexpr int RPS = 256 / TPR;
    extern __shared__ float smem[];
    float* logit = smem;
    float* red = smem + a.C;
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const int L = a.L, C = a.C;
    const int t = threadIdx.x, cc = t % TPR, r0 = t / TPR;
    const int first = chunk * C;
    const bf16* K = static_cast<const bf16*>(a.K) + (bg * (size_t)L + first) * D;
    const bf16* V = static_cast<const bf16*>(a.V) + (bg * (size_t)L + first) * D;
    auto load8 = [&](const bf16* base, int r, float out[8]) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(base + (size_t)r * D + cc * 8);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = bf16_lo(w[i]);
            out[2 * i + 1] = bf16_hi(w[i]);
        }
    };
    auto row_sum = [&](float x) {
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) x += __shfl_xor(x, off, 64);
        return x;
    };
    const float sc = a.scale_log2;  // log2(e) / sqrt(d): logits in log2 units
    const float inv_sqrt_d = sc / kLog2e;
    const size_t cv = (bg * (size_t)a.n_chunks + chunk) * D + cc * 8;  // this thread's features of the chunk
    const size_t kv = bg * (size_t)a.n_chunks * C + first;             // the chunk's first key
    float kh[8] = {0, 0, 0, 0, 0, 0, 0, 0}, gvh[8], dkh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    // summary gradients: sums of the partials of the query-range splits,
    // formed once per feature (threads t < 2 D / 4: four features of dK^ or
    // dV^ each) and shared through LDS
    float* gsh = smem + ((a.C + summary_red_floats<D>() + 3) & ~3);  // [dK^ | dV^], 2 D floats, 16-B aligned
    if (t < 2 * D / 4) {
        const float* src = (t < D / 4 ? a.dKs_w : a.dVs_w) + (bg * (size_t)a.n_chunks + chunk) * D + (t % (D / 4)) * 4;
        const size_t slot = (size_t)a.B * a.Hkv * a.n_chunks * D;
        floatx4 acc4 = *reinterpret_cast<const floatx4*>(src);
        // unrolled to the maximum split count so that the loads are in flight together
#pragma unroll
        for (int sp = 1; sp < kMaxBwdSplits; ++sp)
            if (sp < a.n_split) acc4 += *reinterpret_cast<const floatx4*>(src + sp * slot);
        *reinterpret_cast<floatx4*>(gsh + t * 4) = acc4;
    }
    __syncthreads();
    float gkh[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        gkh[i] = gsh[cc * 8 + i];
        gvh[i] = gsh[D + cc * 8 + i];
    }
    // khat = mean key
    for (int r = r0; r < C; r += RPS) {
        float k[8];
        load8(K, r, k);
#pragma unroll
        for (int i = 0; i < 8; ++i) kh[i] += k[i];
    }
    reduce_rows8<TPR>(kh, red);
#pragma unroll
    for (int i = 0; i < 8; ++i) kh[i] *= 1.f / (float)C;
    // a_j and their max
    float mx = -INFINITY;
    for (int r = r0; r < C; r += RPS) {
        float k[8];
        load8(K, r, k);
        float x = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) x += kh[i] * k[i];
        x = row_sum(x) * sc;
        if (cc == 0) logit[r] = x;
        mx = fmaxf(mx, x);
    }
    const float amax = block_max(mx, red);  // also orders the logit writes before the reads
    // vhat = sum_j b_j v_j (unnormalized) and the denominator
    float vh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
    for (int r = r0; r < C; r += RPS) {
        float v[8];
        load8(V, r, v);
        const float p = fast_exp2(logit[r] - amax);
        psum += p;
#pragma unroll
        for (int i = 0; i < 8; ++i) vh[i] += p * v[i];
    }
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) psum += __shfl_xor(psum, off, 64);
    if ((t & 63) == 0) red[5 * TPR * 8 + (t >> 6)] = psum;
    __syncthreads();
    const float inv_den = 1.f / (red[5 * TPR * 8] + red[5 * TPR * 8 + 1] + red[5 * TPR * 8 + 2] + red[5 * TPR * 8 + 3]);
    __syncthreads();
    reduce_rows8<TPR>(vh, red);
    // dvhat . vhat
    float x = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) x += gvh[i] * vh[i] * inv_den;
    const float gvv = row_sum(x);
    // b_j and da_j = b_j (dvhat . v_j - dvhat . vhat); dkhat = dK^_c + sum_j da_j k_j / sqrt(d)
    for (int r = r0; r < C; r += RPS) {
        float v[8], k[8];
        load8(V, r, v);
        load8(K, r, k);
        float y = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) y += gvh[i] * v[i];
        y = row_sum(y);
        const float bj = fast_exp2(logit[r] - amax) * inv_den;
        const float da = bj * (y - gvv);
        if (cc == 0) {
            a.da_w[kv + r] = da;
            a.bw_w[kv + r] = bj;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) dkh[i] += da * k[i];
    }
    reduce_rows8<TPR>(dkh, red);  // its barriers also order every thread's reads of slot 0 before the write
    if (t < TPR) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a.khat_w[cv + i] = kh[i];
            a.dkhat_w[cv + i] = gkh[i] + dkh[i] * inv_sqrt_d;
            a.dVs_w[cv + i] = gvh[i];  // the total dvhat, for the window tiles
        }
    }
}

// Register-resident variant for chunks of exactly ROWS * RPS rows: every
// thread loads its key and value rows once, and the passes over the chunk
// run on registers (one memory latency per chunk instead of one per pass).
template <int D, int ROWS>
__global__ __launch_bounds__(256) void bwd_summary_kernel_reg(BwdParams a) {
    constexpr int TPR = D / 8;
    constexpr int RPS = 256 / TPR;
    constexpr int C = ROWS * RPS;
    __shared__ float red[summary_red_floats<D>()];
    __shared__ __attribute__((aligned(16))) float gsh[2 * D];  // [dK^ | dV^] of the chunk
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const int L = a.L;
    const int t = threadIdx.x, cc = t % TPR, r0 = t / TPR;
    const int first = chunk * C;
    const bf16* K = static_cast<const bf16*>(a.K) + (bg * (size_t)L + first + r0) * D + cc * 8;
    const bf16* V = static_cast<const bf16*>(a.V) + (bg * (size_t)L + first + r0) * D + cc * 8;
    // read once: non-temporal loads (measured 183 -> 168 us on the LLM workload)
    u32x4 kw[ROWS], vw[ROWS];
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        kw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(K + (size_t)i * RPS * D));
        vw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(V + (size_t)i * RPS * D));
    }
    auto unpack = [&](const u32x4& w, float out[8]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[2 * e] = bf16_lo(w[e]);
            out[2 * e + 1] = bf16_hi(w[e]);
        }
    };
    auto row_sum = [&](float x) {
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) x += __shfl_xor(x, off, 64);
        return x;
    };
    const float sc = a.scale_log2;  // log2(e) / sqrt(d): logits in log2 units
    const float inv_sqrt_d = sc / kLog2e;
    // summary gradients: sums of the partials of the query-range splits
    if (t < 2 * D / 4) {
        const float* src = (t < D / 4 ? a.dKs_w : a.dVs_w) + (bg * (size_t)a.n_chunks + chunk) * D + (t % (D / 4)) * 4;
        const size_t slot = (size_t)a.B * a.Hkv * a.n_chunks * D;
        floatx4 acc4 = *reinterpret_cast<const floatx4*>(src);
#pragma unroll
        for (int sp = 1; sp < kMaxBwdSplits; ++sp)
            if (sp < a.n_split) acc4 += *reinterpret_cast<const floatx4*>(src + sp * slot);
        *reinterpret_cast<floatx4*>(gsh + t * 4) = acc4;
    }
    // khat = mean key
    float kh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
#pragma unroll
        for (int e = 0; e < 8; ++e) kh[e] += k[e];
    }
    reduce_rows8<TPR>(kh, red);  // its barriers also publish gsh
#pragma unroll
    for (int e = 0; e < 8; ++e) kh[e] *= 1.f / (float)C;
    float gkh[8], gvh[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        gkh[e] = gsh[cc * 8 + e];
        gvh[e] = gsh[D + cc * 8 + e];
    }
    // logits (log2 units) and their max
    float sl[ROWS];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) x += kh[e] * k[e];
        sl[i] = row_sum(x) * sc;
        mx = fmaxf(mx, sl[i]);
    }
    const float amax = block_max(mx, red);
    // vhat = sum_j b_j v_j (unnormalized) and the denominator
    float vh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float v[8];
        unpack(vw[i], v);
        sl[i] = fast_exp2(sl[i] - amax);
        psum += sl[i];
#pragma unroll
        for (int e = 0; e < 8; ++e) vh[e] += sl[i] * v[e];
    }
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) psum += __shfl_xor(psum, off, 64);
    if ((t & 63) == 0) red[5 * TPR * 8 + (t >> 6)] = psum;
    __syncthreads();
    const float inv_den = 1.f / (red[5 * TPR * 8] + red[5 * TPR * 8 + 1] + red[5 * TPR * 8 + 2] + red[5 * TPR * 8 + 3]);
    __syncthreads();
    reduce_rows8<TPR>(vh, red);
    // dvhat . vhat
    float x = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) x += gvh[e] * vh[e] * inv_den;
    const float gvv = row_sum(x);
    // b_j, da_j = b_j (dvhat . v_j - dvhat . vhat); dkhat = dK^_c + sum_j da_j k_j / sqrt(d)
    const size_t kv = bg * (size_t)a.n_chunks * C + first + r0;
    float dkh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float v[8], k[8];
        unpack(vw[i], v);
        unpack(kw[i], k);
        float y = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) y += gvh[e] * v[e];
        y = row_sum(y);
        const float bj = sl[i] * inv_den;
        const float da = bj * (y - gvv);
        if (cc == 0) {
            a.da_w[kv + (size_t)i * RPS] = da;
            a.bw_w[kv + (size_t)i * RPS] = bj;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) dkh[e] += da * k[e];
    }
    reduce_rows8<TPR>(dkh, red);
    if (t < TPR) {
        const size_t cv = (bg * (size_t)a.n_chunks + chunk) * D + cc * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            a.khat_w[cv + e] = kh[e];
            a.dkhat_w[cv + e] = gkh[e] + dkh[e] * inv_sqrt_d;
            a.dVs_w[cv + e] = gvh[e];  // the total dvhat, for the window tiles
        }
    }
}

// The same per-chunk pass with one wave per chunk: lane (r0, cc) holds
// features cc*8 .. cc*8+7 of rows r0, r0 + RPS, ... (RPS = 64 / (D / 8)), and
// every reduction is a cross-lane shuffle (no workgroup barrier), so many
// chunks' loads are in flight per CU.  The summary gradients are summed over
// the query-range splits by each lane for its own features.
template <int D, int ROWS>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(ROWS >= 16 ? 2 : 1))) void bwd_summary_kernel_wave(BwdParams a) {
    constexpr int TPR = D / 8;
    constexpr int RPS = 64 / TPR;
    constexpr int C = ROWS * RPS;
    const int chunk = blockIdx.x;
    const size_t bg = blockIdx.y;
    const int L = a.L;
    const int t = threadIdx.x, cc = t % TPR, r0 = t / TPR;
    const int first = chunk * C;
    const bf16* K = static_cast<const bf16*>(a.K) + (bg * (size_t)L + first + r0) * D + cc * 8;
    const bf16* V = static_cast<const bf16*>(a.V) + (bg * (size_t)L + first + r0) * D + cc * 8;
    u32x4 kw[ROWS], vw[ROWS];
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        kw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(K + (size_t)i * RPS * D));
        vw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(V + (size_t)i * RPS * D));
    }
    // summary gradients of this lane's features: sums of the split partials
    // (at most kMaxBwdSplits); row group r0 loads splits r0, r0 + RPS, ...,
    // all in flight together, and the row groups' sums are added across lanes
    float gkh[8], gvh[8];
    {
        static_assert(kMaxBwdSplits % RPS == 0, "splits spread evenly over the row groups");
        const size_t off = (bg * (size_t)a.n_chunks + chunk) * D + cc * 8;
        const size_t slot = (size_t)a.B * a.Hkv * a.n_chunks * D;
        floatx4 k0 = {0.f, 0.f, 0.f, 0.f}, k1 = k0, v0 = k0, v1 = k0;
#pragma unroll
        for (int q = 0; q < kMaxBwdSplits / RPS; ++q) {
            const int sp = r0 + q * RPS;
            if (sp < a.n_split) {
                k0 += *reinterpret_cast<const floatx4*>(a.dKs_w + off + sp * slot);
                k1 += *reinterpret_cast<const floatx4*>(a.dKs_w + off + sp * slot + 4);
                v0 += *reinterpret_cast<const floatx4*>(a.dVs_w + off + sp * slot);
                v1 += *reinterpret_cast<const floatx4*>(a.dVs_w + off + sp * slot + 4);
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            gkh[e] = k0[e];
            gkh[4 + e] = k1[e];
            gvh[e] = v0[e];
            gvh[4 + e] = v1[e];
        }
    }
    auto unpack = [](const u32x4& w, float out[8]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[2 * e] = bf16_lo(w[e]);
            out[2 * e + 1] = bf16_hi(w[e]);
        }
    };
    // over the lanes of one row (its TPR feature groups)
    auto row_sum = [](float x) {
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) x += __shfl_xor(x, off, 64);
        return x;
    };
    // over the lanes holding the same features (the row groups)
    auto rows_sum = [](float x) {
#pragma unroll
        for (int off = TPR; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
        return x;
    };
    const float sc = a.scale_log2;  // log2(e) / sqrt(d): logits in log2 units
    const float inv_sqrt_d = sc / kLog2e;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        gkh[e] = rows_sum(gkh[e]);
        gvh[e] = rows_sum(gvh[e]);
    }
    // khat = mean key
    float kh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
#pragma unroll
        for (int e = 0; e < 8; ++e) kh[e] += k[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) kh[e] = rows_sum(kh[e]) * (1.f / (float)C);
    // logits (log2 units) and their max
    float sl[ROWS];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) x += kh[e] * k[e];
        sl[i] = row_sum(x) * sc;
        mx = fmaxf(mx, sl[i]);
    }
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    // vhat = sum_j b_j v_j (unnormalized), the denominator, and dvhat . v_j
    // (V is not needed after this loop)
    float vh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float psum = 0.f;
    float yv[ROWS];
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float v[8];
        unpack(vw[i], v);
        sl[i] = fast_exp2(sl[i] - mx);
        psum += sl[i];
        float y = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            vh[e] += sl[i] * v[e];
            y += gvh[e] * v[e];
        }
        yv[i] = row_sum(y);
    }
    const float inv_den = 1.f / rows_sum(psum);
    // dvhat . vhat
    float x = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) x += gvh[e] * rows_sum(vh[e]) * inv_den;
    const float gvv = row_sum(x);
    // b_j, da_j = b_j (dvhat . v_j - dvhat . vhat); dkhat = dK^_c + sum_j da_j k_j / sqrt(d)
    const size_t kv = bg * (size_t)a.n_chunks * C + first + r0;
    float dkh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
        float k[8];
        unpack(kw[i], k);
        const float bj = sl[i] * inv_den;
        const float da = bj * (yv[i] - gvv);
        if (cc == 0) {
            a.da_w[kv + (size_t)i * RPS] = da;
            a.bw_w[kv + (size_t)i * RPS] = bj;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) dkh[e] += da * k[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) dkh[e] = rows_sum(dkh[e]);
    if (r0 == 0) {
        // every lane has read the split partials (slot 0 included) above
        const size_t cv = (bg * (size_t)a.n_chunks + chunk) * D + cc * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            a.khat_w[cv + e] = kh[e];
            a.dkhat_w[cv + e] = gkh[e] + dkh[e] * inv_sqrt_d;
            a.dVs_w[cv + e] = gvh[e];  // the total dvhat, for the window tiles
        }
    }
}

}  // namespace

template <int D, int VAR>
hipError_t launch_backward_var(const BwdParams& p, hipStream_t stream) {
    // dQ, and the row dots D = dO . O the dK/dV kernels read
    constexpr int POS = kBwdWaves * 16 * kDqColBlocks;
    const int n_pt = (p.L + POS - 1) / POS;
    hipLaunchKernelGGL((bwd_dq_kernel<D, kDqColBlocks, kDqNS, kDqWpe, VAR>), dim3(p.B * p.H * n_pt),
                       dim3(kBwdWaves * 64), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int KT = kBwdWaves * 16;
    if (p.n_chunks > 0) {
        // summary gradients, then their per-chunk and per-key factors
        const int st = (p.n_chunks + KT - 1) / KT * p.n_split;
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, true, VAR>), dim3(p.B * p.Hkv * st), dim3(kBwdWaves * 64), 0, stream,
                           p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        constexpr int RPS = 256 / (D / 8);
        constexpr int RPW = 64 / (D / 8);  // rows per sweep of one wave
        const dim3 grid(p.n_chunks, p.B * p.Hkv);
        // one wave per chunk when the chunk is 4, 8 or 16 rows per lane
        const int wrows = p.C % RPW == 0 ? p.C / RPW : 0;
        if (wrows == 4 || wrows == 8 || wrows == 16) {
            if (wrows == 4) hipLaunchKernelGGL((bwd_summary_kernel_wave<D, 4>), grid, dim3(64), 0, stream, p);
            if (wrows == 8) hipLaunchKernelGGL((bwd_summary_kernel_wave<D, 8>), grid, dim3(64), 0, stream, p);
            if (wrows == 16) hipLaunchKernelGGL((bwd_summary_kernel_wave<D, 16>), grid, dim3(64), 0, stream, p);
        } else switch (p.C % RPS == 0 ? p.C / RPS : 0) {
            case 1: hipLaunchKernelGGL((bwd_summary_kernel_reg<D, 1>), grid, dim3(256), 0, stream, p); break;
            case 2: hipLaunchKernelGGL((bwd_summary_kernel_reg<D, 2>), grid, dim3(256), 0, stream, p); break;
            case 4: hipLaunchKernelGGL((bwd_summary_kernel_reg<D, 4>), grid, dim3(256), 0, stream, p); break;
            case 8: hipLaunchKernelGGL((bwd_summary_kernel_reg<D, 8>), grid, dim3(256), 0, stream, p); break;
            default: {
                const size_t lds = (size_t)(((p.C + summary_red_floats<D>() + 3) & ~3) + 2 * D) * sizeof(float);
                hipLaunchKernelGGL((bwd_summary_kernel<D>), grid, dim3(256), lds, stream, p);
            }
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const int wt = (p.L + KT - 1) / KT;
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, false, VAR>), dim3(p.B * p.Hkv * wt), dim3(kBwdWaves * 64), 0, stream, p);
    return hipGetLastError();
}

template <int D>
hipError_t launch_backward(const BwdParams& p, hipStream_t stream) {
    switch (p.window) {
        case kWinChunkAligned: return launch_backward_var<D, kWinChunkAligned>(p, stream);
        case kWinBlocked: return launch_backward_var<D, kWinBlocked>(p, stream);
        case kWinNonCausal: return launch_backward_var<D, kWinNonCausal>(p, stream);
        default: return launch_backward_var<D, kWinSliding>(p, stream);
    }
}

template hipError_t launch_backward<64>(const BwdParams&, hipStream_t);
template hipError_t launch_backward<128>(const BwdParams&, hipStream_t);

}  // namespace eva
