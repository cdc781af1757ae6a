// Internal launch interface between the C ABI layer (eva_api.cpp) and the
// kernel translation units.  Host-visible; no torch types anywhere.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace eva {

// Waves per prefill workgroup; each wave owns 32 query columns.
constexpr int kPrefillWaves = 8;
// Pipelined bf16 prefill: 16-column blocks per wave (32 query columns), and
// waves per workgroup of its two configurations: 8 waves on 64-key blocks
// (one workgroup per CU), or 4 waves on 32-key blocks (two workgroups per CU,
// whose prologues and barriers overlap; half the positions per tile).  The
// narrow one is used when every kv head has one query head, and for windows
// of up to 512 keys, where a workgroup's prologue is a large part of its time
// (measured on MI355X: 429 vs 452 us at W 512, 704 vs 694 us at W 1024).
constexpr int kMfmaColBlocks = 2;
constexpr int kMfmaWavesWide = 8;
constexpr int kMfmaWavesNarrow = 4;
inline bool prefill_mfma_narrow(int G, int W) { return G == 1 || W <= 512; }

struct PrefillParams {
    const void* Q;
    const void* K;
    const void* V;
    const void* Ks;  // [B][Hkv][n_chunks][d]
    const void* Vs;
    void* O;
    int B, H, Hkv, L, W, C, n_chunks;
    int G;            // H / Hkv
    int Gt;           // heads packed per workgroup: gcd(G, kPrefillWaves)
    int n_hg;         // G / Gt
    int pos_per_wg;   // 32 * kPrefillWaves / Gt
    int n_pos_tiles;  // ceil(L / pos_per_wg)
    int n_tiles;      // B * Hkv * n_hg * n_pos_tiles
    float scale_log2; // log2(e) / sqrt(d)
    float log2C;      // log2(C): the ln C summary offset in log2 units
    int window;       // window variant (kWin* in eva_device.hpp)
    float* lse;       // optional [B][H][L]: natural log of each row's softmax denominator
    void* O_lo;       // optional, bf16 only, [B][H][L][d]: the output's rounding residual
                      // bf16(o - bf16(o)), so that O + O_lo carries o to ~16 bits
};

template <int D, typename T>
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream);

// Backward of the bf16 prefill (any window variant).  Device pointers; the fp32
// scratch (Dv, dK_w, dV_w, dKs_w, dVs_w) comes from the caller's workspace.
struct BwdParams {
    const void* Q;
    const void* K;
    const void* V;
    const void* Ks;  // [B][Hkv][n_chunks][d], the forward's summaries
    const void* Vs;
    const void* O;
    const void* O_lo;  // optional [B][H][L][d]: the forward's output residual (D = dO . (O + O_lo))
    const void* dO;
    const float* lse;  // [B][H][L], natural log of each row's softmax denominator
    void* dQ;
    void* dK;
    void* dV;
    float* Dv;       // [B][H][L]   dO . O
    float* dKs_w;    // [n_split][B][Hkv][n_chunks][d]   partial gradients of the summary keys / values
    float* dVs_w;    //   (slot 0 of dVs_w holds their sum once the per-chunk pass ran)
    float* khat_w;   // [B][Hkv][n_chunks][d]   mean key of each chunk
    float* dkhat_w;  // [B][Hkv][n_chunks][d]   total gradient of that mean key
    float* da_w;     // [B][Hkv][n_chunks * C]  gradient of each key's chunk-softmax logit
    float* bw_w;     // [B][Hkv][n_chunks * C]  each key's chunk-softmax weight
    int B, H, Hkv, L, W, C, n_chunks;
    int n_split;       // query-range splits of each summary-key tile
    float scale_log2;  // log2(e) / sqrt(d)
    float log2C;
    int window;        // window variant (kWin* in eva_device.hpp)
};

// Splits of the query range of each summary-key tile of the backward (a
// function of the shapes only, so that the workspace size can use it).
constexpr int kMaxBwdSplits = 16;  // query-range splits of a summary tile in the backward
inline int bwd_summary_splits(long long B, long long Hkv, long long L, long long C, long long G) {
    const long long tiles = B * Hkv * ((L / C + 63) / 64);
    if (tiles <= 0) return 1;
    long long s = (2048 + tiles - 1) / tiles;              // about 2048 workgroups
    const long long by_len = ((L + 31) / 32) * G / 8;      // at least ~8 query blocks each
    if (s > by_len) s = by_len;
    if (s > kMaxBwdSplits) s = kMaxBwdSplits;
    return s < 1 ? 1 : (int)s;
}

template <int D>
hipError_t launch_backward(const BwdParams& p, hipStream_t stream);

// bf16 only; tile geometry for the configuration prefill_mfma_narrow(G) picks.
template <int D>
hipError_t launch_prefill_mfma(const PrefillParams& p, hipStream_t stream);

// Chunk summaries; with eps (fp32 [BH][L / C][D]) the stochastic
// random-feature variant with rf_scale = lambda * d^(1/4).
template <int D, typename T>
hipError_t launch_summaries(const void* K, const void* V, void* Ks, void* Vs, int BH, int L, int C,
                            const float* eps, float rf_scale, hipStream_t stream);

// eps [n_seq][n_chunks][D]: the counter-based normal draws (rf_normals4) of
// every chunk of every sequence-head.
template <int D>
hipError_t launch_rf_noise(float* eps, int n_seq, int n_chunks, unsigned long long seed, hipStream_t stream);

struct CacheView {
    int B, H, Hkv, W, C, R, S_max;
    int window;  // causal window variant (kWinSliding / kWinChunkAligned / kWinBlocked)
    // summaries built during decode: stochastic random-feature ones (rf != 0,
    // rf_scale = lambda * d^(1/4), noise from rf_normals4 with rf_seed) or
    // the deterministic ones
    int rf;
    float rf_scale;
    unsigned long long rf_seed;
    long long n_tok;
    void* k_ring;
    void* vt_ring;
    void* k_sum;
    void* vt_sum;
};

// Per-sequence state of a ragged cache, all in device memory.
struct RaggedState {
    int* n_tok;         // [B] tokens held by each sequence
    int* arrive;        // [B] arrival counters of the append kernel (zero between launches)
    const int* active;  // [B] nonzero = the sequence takes part in this step; nullptr = all
    int max_tok;        // most tokens a sequence may hold
};

// Copy the last min(L, R) positions of K/V into the ring and the L / C
// summaries (row-major Ks/Vs) into the cache arrays.  With `lens` (device
// [B], ragged caches) sequence b uses its own length min(lens[b], L,
// r.max_tok) instead of L and the kernel also sets r.n_tok / r.arrive.
template <int D, typename T>
hipError_t launch_cache_fill(const CacheView& c, const void* K, const void* V, const void* Ks, const void* Vs,
                             int L, const int* lens, const RaggedState& r, hipStream_t stream);

// Build summary `s_new` from ring rows (when s_new >= 0), then write the token
// at position p = c.n_tok.
// Append the token at position p (uniform cache): builds the summary of the
// chunk the token completes, then writes the token.
template <int D, typename T>
hipError_t launch_cache_append(const CacheView& c, const void* k_new, const void* v_new, int p, hipStream_t stream);

// Ragged append: every (b, kv head) workgroup reads p = r.n_tok[b] itself,
// builds the summary that becomes due at p, writes the token, and the last
// of the sequence's H_kv workgroups advances r.n_tok[b].
template <int D, typename T>
hipError_t launch_rcache_append(const CacheView& c, const RaggedState& r, const void* k_new, const void* v_new,
                                hipStream_t stream);

struct DecodeParams {
    CacheView c;
    const void* q;  // [B][H][d]
    void* o;        // [B][H][d]
    float* ws;      // split partials or nullptr
    int p;          // position of the query (n_tok - 1)
    int n_sum;      // visible summaries s(p)
    int win_lo;     // first window position
    int n_sum_chunks;  // 32-row chunks of summaries
    int n_win_chunks;  // 32-slot chunks of the ring touched by the window
    int first_win_chunk;
    int splits;     // workgroups per (b, kv head, head group)
    int n_hg;       // head groups of 16 per kv head
    int G;
    float scale_log2;
    float log2C;
    // ragged caches: per-sequence counts in device memory (nullptr for a
    // uniform cache, whose geometry is the host-computed fields above)
    int* n_tok;
    const int* active;
    int max_tok;
    // fused append + decode: the appended token [B][H_kv][d] (nullptr for a
    // plain decode); ragged caches also count arrivals per sequence
    const void* k_new;
    const void* v_new;
    int* arrive;
    int arrivals;  // workgroups per sequence that arrive: splits * H_kv * n_hg + H_kv
};

template <int D, typename T>
hipError_t launch_decode(const DecodeParams& p, hipStream_t stream);

// Fixed device array for the split partials of the allocation-free fused
// decode step: 6.25 MiB, enough for any cache (splits happen only for fewer
// than 256 (b, kv head, head group) units, and then units * splits < 256 +
// 512, each taking 16 * (d + 2) floats).  decode_scratch returns its address
// on the device of `stream` (looked up once per device).
constexpr size_t kDecodeScratchBytes = (size_t)6400 * 1024;
hipError_t decode_scratch(hipStream_t stream, float** out);

}  // namespace eva
