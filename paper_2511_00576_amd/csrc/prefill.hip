// Fused window + summary EVA prefill for gfx950: two-phase kernel, built for
// fp32 (the bf16 path runs the pipelined kernel of prefill_mfma.hip; the
// template keeps its bf16 branches, which that kernel superseded).
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
// round trip) into an NS-deep ring of LDS stages; block j+NS-1 is requested
// while block j is computed, with one barrier per block and an explicit
// vmcnt wait for exactly the block about to be read.  Rows are stored
// unpadded with an XOR swizzle of their 16-B chunks, chosen so that the
// 16-B K-fragment reads and the transposing V reads hit distinct banks.
#include <type_traits>

#include "eva_device.hpp"
#include "eva_kernels.hpp"

namespace eva {

namespace {

constexpr int kBN = 64;      // keys per block
constexpr int kQW = 32;      // query columns per wave
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units)

template <int D, typename T, int NW>
struct PCfg {
    static constexpr bool BF = sizeof(T) == 2;
    static constexpr int ROWB = D * (int)sizeof(T);      // bytes per row
    static constexpr int CPR = ROWB / 16;                // 16-B chunks per row
    static constexpr int VEC = 16 / (int)sizeof(T);      // elements per chunk
    static constexpr int BLK = kBN * ROWB;               // bytes per 64-row block
    static constexpr int NI = BLK / 1024 / NW;           // DMA instructions / wave / array
    static_assert(NI >= 1, "block too small for the workgroup");
    static constexpr int NI_TOTAL = 2 * NI;              // K and V
};

// Chunk swizzles (position = logical chunk ^ swz(row)).  K rows are read as
// 16-B fragments by 16 lanes holding 16 consecutive rows; V rows (bf16) by
// the transposing read, 4 lanes x 8 B on each of 4-8 consecutive rows; V rows
// (fp32) by scalar reads, 16 lanes on each of 4 rows spaced 4 apart.
template <int CPR>
__device__ __forceinline__ int swz_k(int r) {
    return CPR >= 16 ? (r & 15) : ((r >> 1) & 7);
}
template <int CPR, bool BF>
__device__ __forceinline__ int swz_v(int r) {
    if constexpr (BF) return CPR >= 16 ? 2 * (r & 7) : 2 * ((r >> 1) & 3);
    return 4 * ((r >> 2) & 3);
}

template <typename T> struct QFrag;
template <> struct QFrag<bf16> { typedef bf16x8 type; };
template <> struct QFrag<float> { typedef floatx4 type; };

// s_waitcnt immediate: vmcnt(n), lgkmcnt(0), expcnt untouched.
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(N < 64, "vmcnt field is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// One global_load_lds_dwordx4: every lane moves 16 B from base + voff to
// LDS address M0 + 16 * lane.  Issued as inline asm on purpose: the compiler
// cannot see the LDS write, so it does not drain the whole prefetch queue
// (vmcnt(0)) before every later LDS read; the kernel waits for exactly the
// block it is about to read with an explicit vmcnt.  (Waits the compiler
// derives for its own loads only become more conservative: vmcnt retires in
// order.)
__device__ __forceinline__ void lds_dma16(const void* base, unsigned voff, const void* lds_dst) {
    const unsigned m0 =
        __builtin_amdgcn_readfirstlane((unsigned)(size_t)(__attribute__((address_space(3))) const void*)lds_dst);
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(m0) : "memory");
}

// VAR: window variant (win_lo / win_hi / sum_lo / sum_hi); masks of edge
// blocks are per element for every variant.
template <int D, typename T, int NW, int NS, int VAR>
__global__ __launch_bounds__(NW * 64) void prefill_kernel(PrefillParams a) {
    typedef PCfg<D, T, NW> Cfg;
    constexpr bool BF = Cfg::BF;
    constexpr int ROWB = Cfg::ROWB, CPR = Cfg::CPR, VEC = Cfg::VEC, BLK = Cfg::BLK, NI = Cfg::NI;
    constexpr int NQF = BF ? D / 32 : D / 16;  // Q fragments per 16-column block
    constexpr int NDB = D / 16;                // 16-feature output blocks

    __shared__ __attribute__((aligned(1024))) unsigned char lds[NS][2][BLK];

    const T* __restrict__ Q = static_cast<const T*>(a.Q);
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
    const T* Kbg = static_cast<const T*>(a.K) + bg * (size_t)L * D;
    const T* Vbg = static_cast<const T*>(a.V) + bg * (size_t)L * D;
    const T* Ksbg = static_cast<const T*>(a.Ks) + bg * (size_t)a.n_chunks * D;
    const T* Vsbg = static_cast<const T*>(a.Vs) + bg * (size_t)a.n_chunks * D;
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
        dma_vcol[i] = (pos ^ swz_v<CPR, BF>(r)) * VEC;
    }
    auto issue = [&](int j) {
        const int st = j % NS;
        const bool is_sum = j < nsb;
        const int base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        const int limit = is_sum ? a.n_chunks : L;
        const T* kb = (is_sum ? Ksbg : Kbg) + (size_t)base * D;
        const T* vb = (is_sum ? Vsbg : Vbg) + (size_t)base * D;
        // rows past the end repeat the last valid row: finite, and masked out
        // (keys beyond every query, summaries beyond every s(n))
        const int last = limit - 1 - base;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int row = min(dma_row[i], last);
            lds_dma16(kb, (unsigned)((row * D + dma_kcol[i]) * (int)sizeof(T)), &lds[st][0][dma_off[i]]);
            lds_dma16(vb, (unsigned)((row * D + dma_vcol[i]) * (int)sizeof(T)), &lds[st][1][dma_off[i]]);
        }
    };

    // ---- per-lane LDS read offsets (bytes within a stage array) ----
    // K fragment (kb, dc): row kb*16 + c16, logical chunk (bf16) dc*4 + g,
    // (fp32) g*(D/16) + f; the swizzle of row kb*16 + c16 depends on c16 only,
    // so kb only adds kb*16*ROWB (an immediate offset).
    constexpr int NKO = BF ? D / 32 : D / 16;
    int k_off[NKO];
#pragma unroll
    for (int f = 0; f < NKO; ++f) {
        const int chunk = BF ? f * 4 + g : g * (D / 16) + f;
        k_off[f] = c16 * ROWB + ((chunk ^ swz_k<CPR>(c16)) << 4);
    }
    // V, bf16 transposing read: lane (g, 4j'+t) names row 4g+j' (+16 half,
    // +32 kc: immediate offsets) and features 4t..4t+3 of feature block db.
    int v_off[NDB];
    {
        const int v_row = g * 4 + (c16 >> 2);
        const int v_t = c16 & 3;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
            v_off[db] = v_row * ROWB + (((db * 2 + (v_t >> 1)) ^ swz_v<CPR, BF>(v_row)) << 4) + (v_t & 1) * 8;
    }

    floatx4 acc[NDB][2];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) acc[db][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    // softmax denominators: bf16 path sums the rounded weights on the matrix
    // cores (all-ones A operand, every output row = the column sum); fp32 path
    // keeps per-lane partial sums
    floatx4 l_acc[2] = {floatx4{0.f, 0.f, 0.f, 0.f}, floatx4{0.f, 0.f, 0.f, 0.f}};
    float l_run[2] = {0.f, 0.f};
    const bf16x8 ones = {(bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f};

    // ---- staggered two-phase schedule ----
    // phase 1(j): S = QK(j) and the deferred O += PV(j-1)  (matrix cores)
    // phase 2(j): mask + online softmax of S -> P(j)         (vector ALU)
    // Waves [0, NW/2) and [NW/2, NW) sit pairwise on the same SIMD and run
    // one phase apart, so at every tick one wave of each pair feeds the
    // matrix cores while the other runs its softmax.  Tick t ends with a
    // workgroup barrier.  Block k is read from tick 2k (K) until tick 2k+3
    // (V, deferred PV of the second group), so the request for block k+AHEAD
    // may go out at tick 2k into the stage of block k+AHEAD-NS if that block's
    // last read, tick 2(k+AHEAD-NS)+3, is before 2k: AHEAD <= NS-2.  (fp32 does
    // its PV inside phase 2 and keeps all waves in step: last read at 2k+1,
    // AHEAD <= NS-1.)
    static_assert(NS >= 3 || !BF, "the deferred PV needs at least three stages");
    const int group = BF ? wave / (NW / 2) : 0;
    floatx4 s[4][2];
    bf16x8 pf[2][2];
    bool s_ready = false, pv_pending = false;

    auto block_of = [&](int j, int& base, bool& is_sum, bool& needed, bool& full) {
        is_sum = j < nsb;
        base = is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        if (is_sum) {
            const int last = base + kBN - 1;
            needed = base < ws_hi || (NC && w_active && last >= wsx_lo && base < a.n_chunks);
            full = last < ws_lo || (NC && base >= wsx_hi && last < a.n_chunks);
        } else {
            needed = w_active && base <= whi_max && base + kBN - 1 >= wlo_min;
            full = base >= wlo_max && base + kBN - 1 <= whi_min;
        }
    };

    // bf16 phase 1 as one straight-line sequence: the deferred PV of the
    // previous block (V from LDS stage vs) interleaved with QK of this block
    // (K from stage ks); each fragment read is issued at least one step (12
    // MFMAs) before its use.  DP/DQ select the parts present, at compile time,
    // so no branch splits the sequence.
    auto phase1_bf16 = [&](auto dp, auto dq, const unsigned char* ks, const unsigned char* vs) {
        constexpr bool DP = decltype(dp)::value, DQ = decltype(dq)::value;
        constexpr int NDC = D / 32;
        bf16x8 kf[2][4];
        bf16x8 vf[3][2];
        auto load_k = [&](int dc, bf16x8 (&f)[4]) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) f[kb] = *reinterpret_cast<const bf16x8*>(ks + k_off[dc] + kb * 16 * ROWB);
        };
        auto load_v = [&](int db, bf16x8 (&vf2)[2]) {
            const unsigned char* vp = vs + v_off[db];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const shortx4 lo = lds_read_tr16(reinterpret_cast<const bf16*>(vp + (kc * 32) * ROWB));
                const shortx4 hi = lds_read_tr16(reinterpret_cast<const bf16*>(vp + (kc * 32 + 16) * ROWB));
                vf2[kc] = __builtin_bit_cast(
                    bf16x8, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1],
                                                                          hi[2], hi[3]});
            }
        };
        if constexpr (DQ) {
            load_k(0, kf[0]);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) s[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
        if constexpr (DP) {
            load_v(0, vf[0]);
            load_v(1, vf[1]);
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) l_acc[cb] = mfma_bf16(ones, pf[kc][cb], l_acc[cb]);
        }
        constexpr int NSTEP = DP ? NDB : NDC;
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) {
            if constexpr (DQ) {
                if (st + 1 < NDC) load_k(st + 1, kf[(st + 1) & 1]);
            }
            if constexpr (DP) {
                if (st + 2 < NDB) load_v(st + 2, vf[(st + 2) % 3]);
            }
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (DP) {
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) acc[st][cb] = mfma_bf16(vf[st % 3][kc], pf[kc][cb], acc[st][cb]);
            }
            if constexpr (DQ) {
                if (st < NDC) {
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int cb = 0; cb < 2; ++cb)
                            s[kb][cb] = mfma_bf16(kf[st & 1][kb], __builtin_bit_cast(bf16x8, qf[cb][st]), s[kb][cb]);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    constexpr int AHEAD = BF ? NS - 2 : NS - 1;
#pragma unroll
    for (int k = 0; k < AHEAD; ++k)
        if (k < nb) issue(k);
    const int n_ticks = 2 * nb + 2;
    for (int t = 0; t < n_ticks; ++t) {
        // even ticks: block t/2 must have landed; the blocks requested after it
        // may stay in flight.  Always: this wave's LDS reads are done.
        asm volatile("" ::: "memory");
        if ((t & 1) == 0) {
            const int later = min(AHEAD - 1, nb - 1 - t / 2);
            if (AHEAD >= 2 && later >= 1)
                wait_vm_lgkm0<(AHEAD >= 2 ? Cfg::NI_TOTAL : 0)>();
            else
                wait_vm_lgkm0<0>();
        } else {
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        }
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        if ((t & 1) == 0 && t / 2 + AHEAD < nb) issue(t / 2 + AHEAD);

        const int ph = t - group;
        if (ph < 0) continue;
        const int j = ph >> 1;

        if ((ph & 1) == 0) {
            // ---------------- phase 1(j) ----------------
            __builtin_amdgcn_s_setprio(1);
            bool qk = false;
            int base_j = 0;
            if (j < nb) {
                bool is_sum, full;
                block_of(j, base_j, is_sum, qk, full);
            }
            s_ready = qk;
            const unsigned char* ks = lds[j % NS][0];
            if constexpr (BF) {
                const unsigned char* vs = lds[(j + NS - 1) % NS][1];
                const std::true_type yes;
                const std::false_type no;
                if (pv_pending && qk)
                    phase1_bf16(yes, yes, ks, vs);
                else if (pv_pending)
                    phase1_bf16(yes, no, ks, vs);
                else if (qk)
                    phase1_bf16(no, yes, ks, vs);
                pv_pending = false;
            } else if (qk) {
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
            }
            __builtin_amdgcn_s_setprio(0);
        } else if (s_ready) {
            // ---------------- phase 2(j) ----------------
            int base;
            bool is_sum, needed, full;
            block_of(j, base, is_sum, needed, full);

            // mask (boundary blocks only), branch-free per element;
            // element (kb, i) of lane (g, c16) is key base + kb*16 + 4g + i
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
                    l_acc[cb] *= alpha;
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
                        if constexpr (!BF) ls += p;
                    }
                if constexpr (!BF) l_run[cb] += ls;
            }

            if constexpr (BF) {
                // P(j) rounded to bf16 for the deferred PV of phase 1(j+1)
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            pf[kc][cb][i] = to_bf16(s[2 * kc][cb][i]);
                            pf[kc][cb][4 + i] = to_bf16(s[2 * kc + 1][cb][i]);
                        }
                pv_pending = true;
            } else {
                // fp32: O^T += V^T P^T right away; element (key kb*16 + 4g + i,
                // feature db*16 + c16), row swizzle depends on g only
                const unsigned char* vs = lds[j % NS][1];
                const int vsw = swz_v<CPR, BF>(g * 4);
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
                            for (int cb = 0; cb < 2; ++cb)
                                acc[db][cb] = mfma_f32(va, s[kb][cb][i], acc[db][cb]);
                        }
                    }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue: O = acc / l ----
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        const float lt = BF ? l_acc[cb][0] : xgroup_sum(l_run[cb]);
        const int n = col_n[cb];
        if (n >= L) continue;
        const float inv = 1.f / lt;
        // natural log of the softmax denominator: sum 2^(x - m_run) = lt
        if (a.lse && g == 0) a.lse[bh * L + n] = (m_run[cb] + __builtin_amdgcn_logf(lt)) * kLn2;
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

template <int D, typename T, int VAR>
void launch_prefill_var(const PrefillParams& p, hipStream_t stream) {
    constexpr int NS = sizeof(T) == 2 ? 4 : 2;
    hipLaunchKernelGGL((prefill_kernel<D, T, kPrefillWaves, NS, VAR>), dim3(p.n_tiles), dim3(kPrefillWaves * 64), 0,
                       stream, p);
}

template <int D, typename T>
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
    switch (p.window) {
        case kWinChunkAligned: launch_prefill_var<D, T, kWinChunkAligned>(p, stream); break;
        case kWinBlocked: launch_prefill_var<D, T, kWinBlocked>(p, stream); break;
        case kWinNonCausal: launch_prefill_var<D, T, kWinNonCausal>(p, stream); break;
        default: launch_prefill_var<D, T, kWinSliding>(p, stream); break;
    }
    return hipGetLastError();
}

template hipError_t launch_prefill<64, float>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill<128, float>(const PrefillParams&, hipStream_t);

}  // namespace eva
