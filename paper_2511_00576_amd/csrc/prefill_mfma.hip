// Fused window + summary EVA prefill for gfx950, bf16: software-pipelined
// waves.
//
// The attention is the one of the fused FlashEVA formulation (section
// "FlashEVA"): one softmax per query over the exact keys of its local window
// and one key per chunk summary that lies fully before the window, the
// summaries carrying a +ln C logit offset.
//
// Work decomposition: a workgroup is NW waves sharing one K/V head; each wave
// owns CW = 16 NCB query columns (NCB MFMA column blocks), so the workgroup
// covers NW CW columns = Gt heads x (NW CW / Gt) positions.  K/V blocks of BN
// rows are staged HBM -> LDS by global_load_lds_dwordx4 into an NS-stage ring
// and read by every wave; one workgroup barrier per block.  Two
// configurations: 8 waves on 64-key blocks (141 KB of LDS, one workgroup per
// CU), and 4 waves on 32-key blocks (77 KB, two workgroups per CU, whose
// barriers and prologues then overlap), used when each kv head serves one
// query head, where its half-size position tiles also waste fewer blocks at
// the window's edges, and for windows of up to 512 keys (prefill_mfma_narrow).
// Either way two waves share each SIMD.
//
// Per wave and block j one straight-line region runs S^T(j+1) = K Q^T and
// then O^T += V^T P^T(j) in two 32-key halves on the matrix cores, with the
// exponentials of S(j) for the half the next product needs interleaved in the
// same instruction stream, so the matrix cores never wait for the softmax of
// the block they multiply.  Softmax runs in log2 units with a lazy running
// maximum: exponentials use the stored maximum, and the cross-lane maximum
// and the rescale of the accumulators only run when some lane sees a score
// more than 2^8 above it.
//
// Masks.  Blocks entirely inside every column's visible range need none.  A
// window block crossing the causal diagonal or the lower window edge gets one
// of twelve bias patterns (0 / -inf, held in LDS) added to each 16 x 16 score
// tile: the pattern depends only on the lane and on W mod 16, the choice per
// tile only on wave-uniform offsets.  Summary blocks straddling s(n) are
// masked per element.
//
// Window variants (template VAR, see win_lo / win_hi / sum_lo / sum_hi): the
// block plan and the per-wave block classification follow each row's window
// [win_lo(n), win_hi(n)] and summary ranges; the sliding window keeps the bias
// patterns, the other variants test window blocks per element as well.  The
// non-causal variant stages every summary block (its rows see the chunks on
// both sides of their block).
#include <type_traits>

#include "eva_device.hpp"
#include "eva_kernels.hpp"

namespace eva {

namespace {

constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units)
constexpr int kNPat = 12;    // bias patterns: 3 lower-edge x 4 upper-edge states

template <int D, int NW, int NCB, int NS, int BN>
struct MCfg {
    static_assert(BN == 32 || BN == 64, "blocks of 32 or 64 keys");
    static constexpr int ROWB = D * 2;         // bytes per row
    static constexpr int CPR = ROWB / 16;      // 16-B chunks per row
    static constexpr int BLK = BN * ROWB;      // bytes per block of BN rows
    static constexpr int NKB = BN / 16;        // 16-key score tiles per block
    static constexpr int NKC = BN / 32;        // 32-key halves of the value product
    static constexpr int NI = BLK / 1024 / NW; // DMA instructions / wave / array
    static_assert(NI >= 1, "block too small for the workgroup");
    static constexpr int NI_TOTAL = 2 * NI;
    static constexpr int NDC = D / 32;         // contraction steps of S = K Q^T
    static constexpr int NDB = D / 16;         // 16-feature output blocks
    static constexpr int CW = 16 * NCB;        // query columns per wave
};

// Chunk swizzles (stored chunk = logical chunk ^ swz(row)): 16-B K fragment
// reads by 16 lanes on 16 consecutive rows, and transposing V reads by 4 lanes
// x 8 B on each of 4 consecutive rows, both land on distinct banks.
template <int CPR>
__device__ __forceinline__ int mswz_k(int r) {
    return CPR >= 16 ? (r & 15) : ((r >> 1) & 7);
}
template <int CPR>
__device__ __forceinline__ int mswz_v(int r) {
    return CPR >= 16 ? 2 * (r & 7) : 2 * ((r >> 1) & 3);
}

// s_waitcnt immediate: vmcnt(n), lgkmcnt(0), expcnt untouched.
template <int N>
__device__ __forceinline__ void mwait_vm_lgkm0() {
    static_assert(N < 64, "vmcnt field is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Lower-edge state of a 16 x 16 tile whose row offset (query - key at lane
// offset zero) is c, a multiple of 16: 0 all valid, 1 none, 2 diagonal.
__device__ __forceinline__ int lower_state(int c) { return c >= 16 ? 0 : (c < 0 ? 1 : 2); }
// Upper-edge state for e = W - 1 - c: 0 all valid, 1 none, 2 / 3 partial with
// e = e1 (>= 0) or e = e1 - 16 (< 0), e1 = (W - 1) mod 16.
__device__ __forceinline__ int upper_state(int e) { return e >= 15 ? 0 : (e < -15 ? 1 : (e >= 0 ? 2 : 3)); }

// LO: also store the output's rounding residual (training forward); a
// separate instantiation, since even an untaken branch for it in the epilogue
// measured 6-8% slower in the 4-wave configuration.
template <int D, int NW, int NCB, int NS, int BN, int WPE, int VAR, bool LO>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void prefill_mfma_kernel(PrefillParams a) {
    typedef MCfg<D, NW, NCB, NS, BN> Cfg;
    constexpr int kBN = BN, NKB = Cfg::NKB, NKC = Cfg::NKC;
    constexpr int ROWB = Cfg::ROWB, CPR = Cfg::CPR, BLK = Cfg::BLK, NI = Cfg::NI;
    constexpr int NDC = Cfg::NDC, NDB = Cfg::NDB, CW = Cfg::CW, NIT = Cfg::NI_TOTAL;
    constexpr int AHEAD = NS - 1;  // blocks requested ahead of the one computed
    static_assert(NS >= 3 && (NS & (NS - 1)) == 0, "ring of a power-of-two number of stages, at least 3");

    __shared__ __attribute__((aligned(1024))) unsigned char lds[NS][2][BLK];
    __shared__ floatx4 pat[kNPat][64];
    __shared__ __attribute__((aligned(1024))) unsigned char dummy[1024];  // sink of requests past the last block

    const int L = a.L, W = a.W, C = a.C;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;

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

    const int h = kvh * a.G + hg * a.Gt + (wave % a.Gt);
    const int n0 = pt * a.pos_per_wg;
    const int p0 = n0 + (wave / a.Gt) * CW;
    const int n_hi = min(n0 + a.pos_per_wg - 1, L - 1);

    // blocks the workgroup stages: summaries [0, s(n_hi)) (non-causal: all),
    // then the window band
    constexpr bool NC = VAR == kWinNonCausal;
    const int nsb = ((NC ? a.n_chunks : sum_lo<VAR>(n_hi, W, C)) + kBN - 1) / kBN;
    const int kb0 = win_lo<VAR>(n0, W, C) / kBN;
    const int nb = nsb + (win_hi<VAR>(n_hi, W, L) / kBN - kb0 + 1);

    // what this wave needs: prefix summaries c < ws_hi (all columns: c < ws_lo),
    // non-causal suffix summaries c >= wsx_lo (all columns: c >= wsx_hi), and
    // window keys in [wlo_min, whi_max] (all columns: [wlo_max, whi_min])
    const bool w_active = p0 < L;
    const int wp_last = min(p0 + CW - 1, L - 1);
    const int ws_hi = w_active ? sum_lo<VAR>(wp_last, W, C) : 0;
    const int ws_lo = sum_lo<VAR>(p0, W, C);
    const int wsx_lo = NC ? sum_hi<VAR>(p0, W, C, L) : 0;
    const int wsx_hi = NC ? sum_hi<VAR>(wp_last, W, C, L) : 0;
    const int wlo_min = win_lo<VAR>(p0, W, C), wlo_max = win_lo<VAR>(wp_last, W, C);
    const int whi_min = win_hi<VAR>(p0, W, L), whi_max = win_hi<VAR>(wp_last, W, L);

    // ---- request plan.  Block j's rows come from the summaries (j < nsb) or
    // from the window band; with the band's base pointer shifted back by nsb
    // blocks both are "base + j blocks", and the rows valid in block j are
    // (limit - 64 j), limit being n_chunks or L shifted the same way.
    const size_t bg = (size_t)b * a.Hkv + kvh;
    const uintptr_t ks_base = (uintptr_t)a.Ks + bg * (size_t)a.n_chunks * ROWB;
    const uintptr_t vs_base = (uintptr_t)a.Vs + bg * (size_t)a.n_chunks * ROWB;
    const uintptr_t kw_base = (uintptr_t)a.K + bg * (size_t)L * ROWB + (uintptr_t)((intptr_t)(kb0 - nsb) * BLK);
    const uintptr_t vw_base = (uintptr_t)a.V + bg * (size_t)L * ROWB + (uintptr_t)((intptr_t)(kb0 - nsb) * BLK);
    const int sum_limit = a.n_chunks;
    const int win_limit = L - (kb0 - nsb) * kBN;
    // per lane: instruction i of this wave fills LDS bytes
    // [(i*NW + wave) * 1024, +1024) of each array; lane -> (row, chunk)
    int dma_row[NI], dma_koff[NI], dma_voff[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int byte = (i * NW + wave) * 1024 + lane * 16;
        const int r = byte / ROWB;
        const int pos = (byte % ROWB) / 16;
        dma_row[i] = r;
        dma_koff[i] = ((pos ^ mswz_k<CPR>(r)) << 4) - r * ROWB;  // added to row * ROWB
        dma_voff[i] = ((pos ^ mswz_v<CPR>(r)) << 4) - r * ROWB;
    }
    // part q of block j's request: K for even q, V for odd q, instruction q/2;
    // blocks past the last one go to a dummy LDS area, so that every wave has
    // the same number of requests in flight at every wait
    struct Req {
        uintptr_t k, v;
        int last;        // last valid row of the block
        unsigned stage;  // LDS byte address of the block's stage
    };
    auto request = [&](int j) {
        Req r;
        const bool sum = j < nsb;
        const bool real = j < nb;
        const uintptr_t off = (uintptr_t)j * BLK;
        r.k = (sum ? ks_base : kw_base) + off;
        r.v = (sum ? vs_base : vw_base) + off;
        r.last = min((sum ? sum_limit : win_limit) - j * kBN, kBN) - 1;
        if (!real) {
            r.k = (uintptr_t)a.K;  // any valid row
            r.v = (uintptr_t)a.V;
            r.last = 0;
        }
        r.stage = real ? (unsigned)(size_t)(__attribute__((address_space(3))) void*)&lds[j & (NS - 1)][0][0]
                       : (unsigned)(size_t)(__attribute__((address_space(3))) void*)dummy;
        return r;
    };
    auto issue_part = [&](const Req& r, int q) {
        const int i = q >> 1;
        const bool is_v = q & 1;
        const int row = min(dma_row[i], r.last);
        const unsigned voff = (unsigned)(row * ROWB + (is_v ? dma_voff[i] : dma_koff[i]) + dma_row[i] * ROWB);
        // the dummy area takes every part at the same address
        const unsigned dst = r.stage == (unsigned)(size_t)(__attribute__((address_space(3))) void*)dummy
                                 ? r.stage
                                 : r.stage + (is_v ? BLK : 0) + (i * NW + wave) * 1024;
        asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(is_v ? r.v : r.k),
                     "{m0}"(__builtin_amdgcn_readfirstlane(dst))
                     : "memory");
    };

    // ---- bias patterns: pattern (lo, up) at lane (g, c16), element i is the
    //      mask of query c16 vs key 4g + i of a tile with the given edge states
    if (VAR == kWinSliding && wave == 0) {
        const int e1 = (W - 1) & 15;
#pragma unroll
        for (int p = 0; p < kNPat; ++p) {
            const int lo = p / 4, up = p % 4;
            floatx4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int x = c16 - 4 * g - i;  // query - key inside the tile
                const bool lo_ok = lo == 0 || (lo == 2 && x >= 0);
                const bool up_ok = up == 0 || (up == 2 && x <= e1) || (up == 3 && x <= e1 - 16);
                v[i] = (lo_ok && up_ok) ? 0.f : -INFINITY;
            }
            pat[p][lane] = v;
        }
    }

    auto col_n = [&](int cb) { return p0 + cb * 16 + c16; };

    // ---- Q fragments (B operand of S^T = K Q^T): features dc*32 + 8g .. +7.
    // Columns past L read row L-1: finite, and their outputs are not stored.
    const bf16* __restrict__ Q = static_cast<const bf16*>(a.Q);
    const size_t bh = (size_t)b * a.H + h;
    bf16x8 qf[NCB][NDC];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const bf16* qrow = Q + (bh * L + (size_t)min(col_n(cb), L - 1)) * D;
#pragma unroll
        for (int f = 0; f < NDC; ++f) qf[cb][f] = *reinterpret_cast<const bf16x8*>(qrow + f * 32 + g * 8);
    }

    // ---- LDS read offsets ----
    // K fragment (kb, dc): row kb*16 + c16, logical chunk dc*4 + g; offset
    // k0 ^ (dc << 6) (kb adds an immediate kb*16*ROWB).  V transposing read:
    // lane (g, 4j'+t) names row 4g+j' (+16 half, +32 kc), features 4t..4t+3
    // of feature block db (logical chunk 2 db + t/2); offset v0 ^ (db << 5).
    const int k0 = c16 * ROWB + ((g ^ mswz_k<CPR>(c16)) << 4);
    int v0;
    {
        const int v_row = g * 4 + (c16 >> 2);
        const int v_t = c16 & 3;
        v0 = v_row * ROWB + (((v_t >> 1) ^ mswz_v<CPR>(v_row)) << 4) + (v_t & 1) * 8;
    }
    auto kfrag = [&](const unsigned char* ks, int kb, int dc) {
        return *reinterpret_cast<const bf16x8*>(ks + (k0 ^ (dc << 6)) + kb * 16 * ROWB);
    };
    auto vfrag = [&](const unsigned char* vs, int db, int kc) {
        const unsigned char* vp = vs + (v0 ^ (db << 5)) + kc * 32 * ROWB;
        const shortx4 lo = lds_read_tr16(reinterpret_cast<const bf16*>(vp));
        const shortx4 hi = lds_read_tr16(reinterpret_cast<const bf16*>(vp + 16 * ROWB));
        return __builtin_bit_cast(
            bf16x8, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
    };

    floatx4 acc[NDB][NCB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[db][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    // running maxima (log2 units, identical on the four lanes of a column) and
    // denominators: row sums of the bf16-rounded weights on the matrix cores
    // (all-ones A operand, every output row holds the column sum)
    // m_neg: -m_run, or 0 while m_run is -inf (a column that has seen no key
    // yet), kept beside it so that each step's exponent offset is one add
    float m_run[NCB], m_neg[NCB];
    floatx4 l_acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        m_run[cb] = -INFINITY;
        m_neg[cb] = 0.f;
        l_acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    const bf16x8 ones = {(bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f};
    // scores of two consecutive blocks.  s1 starts at zero: a wave that needs
    // neither block 0 nor block 1 skips iteration 0, so s1 is first read (as
    // the scores of a block it does not need, whose weights must come out 0)
    // before any product wrote it.
    floatx4 s0[NKB][NCB], s1[NKB][NCB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) s1[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    bf16x8 pf[NKC][NCB];             // P^T of the current block, per 32-key half
    float lm[NCB], alpha[NCB];
    bool pending = false;            // rescale owed to the accumulators

    // block classification for this wave
    struct Blk {
        int base;
        bool is_sum, needed, full;
    };
    auto block_of = [&](int j) {
        Blk k;
        k.is_sum = j < nsb;
        k.base = k.is_sum ? j * kBN : (kb0 + j - nsb) * kBN;
        if (k.is_sum) {
            const int last = k.base + kBN - 1;
            k.needed = k.base < ws_hi || (NC && w_active && last >= wsx_lo && k.base < a.n_chunks);
            k.full = last < ws_lo || (NC && k.base >= wsx_hi && last < a.n_chunks);
        } else {
            k.needed = w_active && k.base <= whi_max && k.base + kBN - 1 >= wlo_min;
            k.full = k.base >= wlo_max && k.base + kBN - 1 <= whi_min;
        }
        return k;
    };
    // window block crossing an edge: every score tile gets its bias pattern
    // added (0 or -inf per element)
    auto add_bias = [&](floatx4 (&sd)[NKB][NCB], int base) {
        const int delta = p0 - base;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int c = delta + 16 * (cb - kb);
                sd[kb][cb] += pat[lower_state(c) * 4 + upper_state(W - 1 - c)][lane];
            }
    };
    auto lane_max = [&](floatx4 (&sc)[NKB][NCB]) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sc[kb][cb][i]);
            lm[cb] = mx;
        }
    };
    // summary block straddling s(n): key base + kb*16 + 4g + i valid iff < s(n)
    // (non-causal: or in [sum_hi(n), n_chunks))
    auto mask_sum = [&](floatx4 (&sc)[NKB][NCB], int base) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const int n = min(col_n(cb), L - 1);
            const int lim = sum_lo<VAR>(n, W, C) - base - g * 4;
            const int lim_x = (NC ? sum_hi<VAR>(n, W, C, L) : 0) - base - g * 4;
            const int lim_n = a.n_chunks - base - g * 4;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int x = kb * 16 + i;
                    const bool ok = x < lim || (NC && x >= lim_x && x < lim_n);
                    sc[kb][cb][i] = ok ? sc[kb][cb][i] : -INFINITY;
                }
        }
    };
    // window block crossing an edge, variants other than sliding: key
    // base + kb*16 + 4g + i valid iff win_lo(n) <= key <= win_hi(n)
    auto mask_win = [&](floatx4 (&sc)[NKB][NCB], int base) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const int n = min(col_n(cb), L - 1);
            const int lo = win_lo<VAR>(n, W, C);
            const unsigned span = (unsigned)(win_hi<VAR>(n, W, L) - lo);
            const int rel0 = base + g * 4 - lo;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    sc[kb][cb][i] = (unsigned)(rel0 + kb * 16 + i) <= span ? sc[kb][cb][i] : -INFINITY;
        }
    };
    auto mask_window = [&](floatx4 (&sc)[NKB][NCB], int base) {
        if constexpr (VAR == kWinSliding)
            add_bias(sc, base);
        else
            mask_win(sc, base);
    };
    // lazy maximum update once the scores of a block are known; returns
    // whether the accumulators must be rescaled by alpha
    auto update_max = [&](float bias) -> bool {
        bool need = false;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) need |= lm[cb] * a.scale_log2 + bias > m_run[cb] + kTau;
        if (__ballot(need) == 0) return false;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const float bm = xgroup_max(lm[cb]) * a.scale_log2 + bias;
            const bool up = bm > m_run[cb] + kTau;
            alpha[cb] = up ? fast_exp2(m_run[cb] - bm) : 1.f;
            m_run[cb] = up ? bm : m_run[cb];
            m_neg[cb] = m_run[cb] == -INFINITY ? 0.f : -m_run[cb];
        }
        return true;
    };
    auto rescale = [&]() {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            l_acc[cb] *= alpha[cb];
#pragma unroll
            for (int db = 0; db < NDB; ++db) acc[db][cb] *= alpha[cb];
        }
    };
    // wait until a block landed (LATER blocks requested after it may stay in
    // flight), then make it visible to the whole workgroup; every wave's
    // reads of the stage about to be refilled are done as well
    auto sync_block = [&](auto later_tag) {
        constexpr int LATER = decltype(later_tag)::value;
        asm volatile("" ::: "memory");
        mwait_vm_lgkm0<LATER * NIT>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };

    // ---- prologue: blocks 0 .. AHEAD-1 requested (after the queries), S^T of
    //      block 0.  The product runs whether or not this wave needs block 0,
    //      so that the wait for the queries sits here on every path.
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) {
        const Req r = request(k);
#pragma unroll
        for (int q = 0; q < NIT; ++q) issue_part(r, q);
    }
    sync_block(std::integral_constant<int, AHEAD - 1>{});  // also the patterns
    Blk kc = block_of(0);
    {
        const unsigned char* ks = lds[0][0];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) s0[kb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        bf16x8 kf[2][4];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) kf[0][kb] = kfrag(ks, kb, 0);
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc) {
            if (dc + 1 < NDC) {
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) kf[(dc + 1) & 1][kb] = kfrag(ks, kb, dc + 1);
            }
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) s0[kb][cb] = mfma_bf16(kf[dc & 1][kb], qf[cb][dc], s0[kb][cb]);
        }
        if (kc.needed) {
            if (kc.is_sum && !kc.full) mask_sum(s0, kc.base);
            if (!kc.is_sum && !kc.full) mask_window(s0, kc.base);
            lane_max(s0);
            update_max(kc.is_sum ? a.log2C : 0.f);  // acc is zero: no rescale owed
        }
    }

    // ---- iteration j: S^T(j+1) and O^T += V^T P^T(j) ----
    auto iteration = [&](auto ph_tag, int j, floatx4 (&sc)[NKB][NCB], floatx4 (&sn)[NKB][NCB]) {
        constexpr int PH = decltype(ph_tag)::value;  // j mod NS: the stages as constants
        // block j+1 landed (the AHEAD-2 blocks after it may stay in flight);
        // the block requested in this iteration refills the stage of block
        // j-1, whose last reads were before this barrier
        sync_block(std::integral_constant<int, AHEAD - 2>{});
        if (pending) {
            rescale();
            pending = false;
        }
        const Req req = request(j + AHEAD);
        const bool has_next = j + 1 < nb;
        Blk kn{0, false, false, true};
        if (has_next) kn = block_of(j + 1);
        const bool do_pv = kc.needed;
        const bool do_qk = has_next && kn.needed;
        const float bias_c = kc.is_sum ? a.log2C : 0.f;
        const unsigned char* ks = lds[(PH + 1) & (NS - 1)][0];
        const unsigned char* vs = lds[PH][1];
        if (!do_pv && !do_qk) {
            // nothing of blocks j, j+1 for this wave: only its share of the request
#pragma unroll
            for (int q = 0; q < NIT; ++q) issue_part(req, q);
            kc = kn;
            return;
        }

        // One straight-line region, as a sequence of steps, each with one LDS
        // operand fragment and the matrix-core work on it:
        //   A (4 NDC steps): S^T(j+1), key tile kb, contraction step dc  | exponentials, half 0 of S(j)
        //   B (NDB steps):   O^T += V^T P^T, feature block db, keys 0..31 | exponentials, half 1 of S(j)
        //   C (NDB steps):   same for keys 32..63                        | lane maxima of S(j+1)
        // Fragments are requested PF steps ahead; a scheduling fence between
        // steps keeps that distance (and the register count) fixed.  The
        // parts of this iteration's request are spread over the region.  The
        // region is the same code whether or not this wave needs block j or
        // j+1 (alternative variants cost the register allocator dearly): a
        // block the wave does not need gets zero weights (offset -inf) in its
        // PV, and scores nobody needs are not used.
        constexpr int NA = NKB * NDC;  // steps of part A
        constexpr int N = NA + NKC * NDB;
        constexpr int PF = 2;          // prefetch distance in steps
        constexpr int EH = NCB * 8;    // exponentials per 32-key half and lane
        constexpr int MV = NCB * NKB * 4;  // scores per block and lane
        float off[NCB];
        const float bias_sel = do_pv ? bias_c : -INFINITY;  // wave-uniform
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) off[cb] = bias_sel + m_neg[cb];
        // P^T half hf: contraction row 8g + e is key (2hf)*16 + 4g + e for
        // e < 4, (2hf+1)*16 + 4g + e - 4 above (the V^T read uses the same order)
        auto ex = [&](int hf, int ef) {
            const int cb = ef / 8, e = ef % 8;
            const float sv = sc[2 * hf + (e >> 2)][cb][e & 3];
            pf[hf][cb][e] = to_bf16(fast_exp2(fmaf(sv, a.scale_log2, off[cb])));
        };
        auto mx = [&](int v) {
            const int cb = v / (NKB * 4), kb = (v % (NKB * 4)) / 4, i = v % 4;
            lm[cb] = fmaxf(lm[cb], sn[kb][cb][i]);
        };
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) lm[cb] = -INFINITY;
        bf16x8 op[PF + 1];  // fragment ring
        auto load = [&](int k) {
            if (k < NA)
                op[k % (PF + 1)] = kfrag(ks, k % NKB, k / NKB);
            else
                op[k % (PF + 1)] = vfrag(vs, (k - NA) % NDB, (k - NA) / NDB);
        };
        auto fetch = [&](int k) {
            if (k + PF < N) load(k + PF);
        };
#pragma unroll
        for (int k = 0; k < PF; ++k) load(k);
#pragma unroll
        for (int q = 0; q < NIT / 2; ++q) issue_part(req, q);
#pragma unroll
        for (int k = 0; k < NA; ++k) {
            fetch(k);
            const int kb = k % NKB, dc = k / NKB;
            const bf16x8 f = op[k % (PF + 1)];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                sn[kb][cb] = mfma_bf16(f, qf[cb][dc], dc == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : sn[kb][cb]);
#pragma unroll
            for (int ef = k * EH / NA; ef < (k + 1) * EH / NA; ++ef) ex(0, ef);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int q = NIT / 2; q < 3 * NIT / 4; ++q) issue_part(req, q);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) l_acc[cb] = mfma_bf16(ones, pf[0][cb], l_acc[cb]);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const int k = NA + db;
            fetch(k);
            const bf16x8 f = op[k % (PF + 1)];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) acc[db][cb] = mfma_bf16(f, pf[0][cb], acc[db][cb]);
            if constexpr (NKC == 2) {
#pragma unroll
                for (int ef = db * EH / NDB; ef < (db + 1) * EH / NDB; ++ef) ex(1, ef);
            } else {
#pragma unroll
                for (int v = db * MV / NDB; v < (db + 1) * MV / NDB; ++v) mx(v);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int q = 3 * NIT / 4; q < NIT; ++q) issue_part(req, q);
        if constexpr (NKC == 2) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) l_acc[cb] = mfma_bf16(ones, pf[NKC - 1][cb], l_acc[cb]);
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
                const int k = NA + NDB + db;
                fetch(k);
                const bf16x8 f = op[k % (PF + 1)];
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) acc[db][cb] = mfma_bf16(f, pf[NKC - 1][cb], acc[db][cb]);
#pragma unroll
                for (int v = db * MV / NDB; v < (db + 1) * MV / NDB; ++v) mx(v);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (do_qk) {
            // boundary blocks: masks after the product, then the lane maxima again
            if (!kn.full) {
                if (kn.is_sum)
                    mask_sum(sn, kn.base);
                else
                    mask_window(sn, kn.base);
                lane_max(sn);
            }
            pending = update_max(kn.is_sum ? a.log2C : 0.f);
        }
        kc = kn;
    };
    // four steps per trip, so that each one's stage indices are constants
    static_assert(NS == 4, "one trip covers the ring");
    typedef std::integral_constant<int, 0> P0;
    typedef std::integral_constant<int, 1> P1;
    typedef std::integral_constant<int, 2> P2;
    typedef std::integral_constant<int, 3> P3;
    int j = 0;
    for (; j + 3 < nb; j += 4) {
        iteration(P0{}, j, s0, s1);
        iteration(P1{}, j + 1, s1, s0);
        iteration(P2{}, j + 2, s0, s1);
        iteration(P3{}, j + 3, s1, s0);
    }
    if (j < nb) iteration(P0{}, j, s0, s1);
    if (j + 1 < nb) iteration(P1{}, j + 1, s1, s0);
    if (j + 2 < nb) iteration(P2{}, j + 2, s0, s1);
    if (pending) rescale();

    // No request may still be writing LDS when the workgroup ends: wait for
    // them before the stores, which need not complete before the end.
    mwait_vm_lgkm0<0>();

    // ---- epilogue: O = acc / l, staged through LDS so that each store
    // instruction writes whole output rows ----
    // Straight from the accumulators a store instruction would write 16
    // pieces of 32 bytes (a row's features 4g .. 4g+3 for 16 rows); measured
    // on MI355X, whole rows take the LLM workload from 347 to 331 us, and the
    // training forward with the residual from 434 to 356 us.  Every wave is
    // done with the ring: it holds the staged rows now (a wave's CW rows with
    // a 32-byte skew between rows, so the fragment writes of one instruction
    // fall in distinct banks).  Stores are non-temporal: nothing here reads
    // the rows again.
    __builtin_amdgcn_s_barrier();
    constexpr int SROW = 2 * D + 32;
    constexpr int LPR = 2 * D / 16;   // lanes per row (16 bytes each)
    constexpr int RPI = 64 / LPR;     // rows per store instruction
    static_assert(NW * CW * SROW <= NS * 2 * BLK, "staged rows fit in the ring");
    unsigned char* const stg = &lds[0][0][0] + wave * CW * SROW;
    float inv[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        inv[cb] = 1.f / l_acc[cb][0];
        const int n = col_n(cb);
        // natural log of the softmax denominator: sum 2^(x - m_run) = l
        if (a.lse && g == 0 && n < L) a.lse[bh * L + n] = (m_run[cb] + __builtin_amdgcn_logf(l_acc[cb][0])) * kLn2;
    }
    // rows p0 + r of this wave's head, r = i RPI + lane / LPR
    auto store_rows = [&](bf16* base) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int i = 0; i < CW / RPI; ++i) {
            const int r = i * RPI + lane / LPR;
            const u32x4 x = *reinterpret_cast<const u32x4*>(stg + r * SROW + (lane % LPR) * 16);
            const int n = p0 + r;
            bf16* dst = base + (bh * L + (size_t)n) * D + (lane % LPR) * 8;
            if (n < L) __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(dst));
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const floatx4 v = acc[db][cb] * inv[cb];
            const u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
            *reinterpret_cast<u32x2*>(stg + (cb * 16 + c16) * SROW + (db * 16 + 4 * g) * 2) = w;
        }
    store_rows(static_cast<bf16*>(a.O));
    if constexpr (LO) {
        // residual of the rounding: what the bf16 output lost
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
                const floatx4 v = acc[db][cb] * inv[cb];
                const u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                const u32x2 r = {pack_bf16x2(v[0] - bf16_lo(w[0]), v[1] - bf16_hi(w[0])),
                                 pack_bf16x2(v[2] - bf16_lo(w[1]), v[3] - bf16_hi(w[1]))};
                *reinterpret_cast<u32x2*>(stg + (cb * 16 + c16) * SROW + (db * 16 + 4 * g) * 2) = r;
            }
        store_rows(static_cast<bf16*>(a.O_lo));
    }
}

}  // namespace

template <int D, int VAR, bool LO = false>
void launch_prefill_mfma_var(const PrefillParams& p, hipStream_t stream) {
    if (prefill_mfma_narrow(p.G, p.W)) {
        // 4 waves x 32 columns, 32-key blocks: 77 KB of LDS, two workgroups per CU
        hipLaunchKernelGGL((prefill_mfma_kernel<D, kMfmaWavesNarrow, kMfmaColBlocks, 4, 32, 2, VAR, LO>),
                           dim3(p.n_tiles), dim3(kMfmaWavesNarrow * 64), 0, stream, p);
    } else {
        // 8 waves x 32 columns, 64-key blocks: 141 KB of LDS, one workgroup per CU
        hipLaunchKernelGGL((prefill_mfma_kernel<D, kMfmaWavesWide, kMfmaColBlocks, 4, 64, 2, VAR, LO>),
                           dim3(p.n_tiles), dim3(kMfmaWavesWide * 64), 0, stream, p);
    }
}

template <int D>
hipError_t launch_prefill_mfma(const PrefillParams& p, hipStream_t stream) {
    if (p.O_lo) {
        // the training forward, keeping the output's rounding residual
        switch (p.window) {
            case kWinChunkAligned: launch_prefill_mfma_var<D, kWinChunkAligned, true>(p, stream); break;
            case kWinBlocked: launch_prefill_mfma_var<D, kWinBlocked, true>(p, stream); break;
            case kWinNonCausal: launch_prefill_mfma_var<D, kWinNonCausal, true>(p, stream); break;
            default: launch_prefill_mfma_var<D, kWinSliding, true>(p, stream); break;
        }
        return hipGetLastError();
    }
    switch (p.window) {
        case kWinChunkAligned: launch_prefill_mfma_var<D, kWinChunkAligned>(p, stream); break;
        case kWinBlocked: launch_prefill_mfma_var<D, kWinBlocked>(p, stream); break;
        case kWinNonCausal: launch_prefill_mfma_var<D, kWinNonCausal>(p, stream); break;
        default: launch_prefill_mfma_var<D, kWinSliding>(p, stream); break;
    }
    return hipGetLastError();
}

template hipError_t launch_prefill_mfma<64>(const PrefillParams&, hipStream_t);
template hipError_t launch_prefill_mfma<128>(const PrefillParams&, hipStream_t);

}  // namespace eva
