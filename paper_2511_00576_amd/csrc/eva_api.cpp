// C ABI of libeva: argument validation, launch geometry, dtype/head-dim
// dispatch and the decode cache's host-side bookkeeping.  Every function
// validates before enqueuing anything and never allocates, frees or
// synchronizes.
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "../../include/eva.h"
#include "eva_device.hpp"
#include "eva_kernels.hpp"

using eva::bf16;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int supported(int d, int dtype) {
    if (dtype != EVA_BF16 && dtype != EVA_F32) return EVA_ERR_UNSUPPORTED;
    if (d != 64 && d != 128) return EVA_ERR_UNSUPPORTED;
    return EVA_OK;
}

// Window variants (eva_window): first exact key of row n, and the number of
// summaries that lie wholly before it.  Non-causal rows also see chunks
// after their block (not needed by the decode path, which is causal).
long long window_lo(int window, long long n, long long W, long long C) {
    switch (window) {
        case EVA_WINDOW_CHUNK_ALIGNED: return (n - W + 1 > 0 ? (n - W + 1) / C : 0) * C;
        case EVA_WINDOW_BLOCKED:
        case EVA_WINDOW_NONCAUSAL: return (n / W) * W;
        default: return n - W + 1 > 0 ? n - W + 1 : 0;
    }
}
int prefix_summaries(int window, long long n, long long W, long long C) {
    return (int)(window_lo(window, n, W, C) / C);
}
// Whether any row of a sequence of L tokens can see a summary (then the
// summary pointers must be valid).
bool any_summary(int window, long long L, long long W, long long C) {
    if (window == EVA_WINDOW_NONCAUSAL) return L / C > 0;
    return prefix_summaries(window, L - 1, W, C) > 0;
}
bool valid_window(int window) { return window >= EVA_WINDOW_SLIDING && window <= EVA_WINDOW_NONCAUSAL; }

int hip_status(hipError_t e) { return e == hipSuccess ? EVA_OK : EVA_ERR_HIP; }

template <typename F>
hipError_t dispatch(int d, int dtype, F&& f) {
    if (dtype == EVA_BF16) {
        if (d == 64) return f(std::integral_constant<int, 64>(), bf16());
        return f(std::integral_constant<int, 128>(), bf16());
    }
    if (d == 64) return f(std::integral_constant<int, 64>(), float());
    return f(std::integral_constant<int, 128>(), float());
}

// Largest C whose logits fit the summary kernel's LDS scratch.
constexpr int kMaxChunk = 8192;
// Longest sequence (L) the entry points take: kernel index arithmetic stays
// in 32 bits with room to spare.
constexpr int kMaxLen = 1 << 30;

int check_cache(const eva_cache* c) {
    if (!c) return EVA_ERR_INVALID;
    if (c->B < 1 || c->H < 1 || c->H_kv < 1 || c->H % c->H_kv != 0 || c->W < 1 || c->C < 1 || c->C > kMaxChunk)
        return EVA_ERR_INVALID;
    int st = supported(c->d, c->dtype);
    if (st != EVA_OK) return st;
    if (!c->k_ring || !c->vt_ring || !c->k_sum || !c->vt_sum) return EVA_ERR_INVALID;
    if (!aligned16(c->k_ring) || !aligned16(c->vt_ring) || !aligned16(c->k_sum) || !aligned16(c->vt_sum))
        return EVA_ERR_INVALID;
    if (c->n_tok < 0) return EVA_ERR_INVALID;
    if (c->n_tok >= kMaxLen) return EVA_ERR_CAPACITY;  // positions stay below 2^30
    if (!valid_window(c->window) || c->window == EVA_WINDOW_NONCAUSAL) return EVA_ERR_INVALID;
    if (c->R < 32 || c->R % 32 != 0 || c->S_max < 32 || c->S_max % 32 != 0) return EVA_ERR_INVALID;
    if ((long long)c->R < (long long)c->W + c->C - 1) return EVA_ERR_CAPACITY;
    if ((long long)c->B * c->H_kv > 65535) return EVA_ERR_UNSUPPORTED;
    if (c->rf != 0 && c->rf != 1) return EVA_ERR_INVALID;
    if (c->rf && (!(c->rf_lambda >= 0.f) || c->rf_lambda > 1e30f)) return EVA_ERR_INVALID;
    return EVA_OK;
}

// lambda * d^(1/4): the noise's weight in the summaries' logit vectors
float rf_scale_of(int rf, float lambda, int d) { return rf ? (float)(lambda * sqrt(sqrt((double)d))) : 0.f; }

eva::CacheView view_of(const eva_cache* c) {
    eva::CacheView v;
    v.B = c->B;
    v.H = c->H;
    v.Hkv = c->H_kv;
    v.W = c->W;
    v.C = c->C;
    v.R = c->R;
    v.S_max = c->S_max;
    v.n_tok = c->n_tok;
    v.window = c->window;
    v.k_ring = c->k_ring;
    v.vt_ring = c->vt_ring;
    v.k_sum = c->k_sum;
    v.vt_sum = c->vt_sum;
    v.rf = c->rf;
    v.rf_scale = rf_scale_of(c->rf, c->rf_lambda, c->d);
    v.rf_seed = c->rf_seed;
    return v;
}

int gcd(int a, int b) {
    while (b) {
        int t = a % b;
        a = b;
        b = t;
    }
    return a;
}

// Split count for decode: enough workgroups to cover the chip when B * H_kv
// is small, never more than one wave per chunk.
int decode_splits(int units, int n_chunks) {
    if (units >= 256) return 1;
    int s = (512 + units - 1) / units;
    int max_s = (n_chunks + 3) / 4;
    if (s > max_s) s = max_s;
    return s < 1 ? 1 : s;
}

int check_rcache(const eva_rcache* c) {
    if (!c) return EVA_ERR_INVALID;
    if (c->B < 1 || c->H < 1 || c->H_kv < 1 || c->H % c->H_kv != 0 || c->W < 1 || c->C < 1 || c->C > kMaxChunk)
        return EVA_ERR_INVALID;
    int st = supported(c->d, c->dtype);
    if (st != EVA_OK) return st;
    if (!c->k_ring || !c->vt_ring || !c->k_sum || !c->vt_sum || !c->n_tok || !c->arrive) return EVA_ERR_INVALID;
    if (c->max_tok > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (!aligned16(c->k_ring) || !aligned16(c->vt_ring) || !aligned16(c->k_sum) || !aligned16(c->vt_sum))
        return EVA_ERR_INVALID;
    if (c->max_tok < 1) return EVA_ERR_INVALID;
    if (!valid_window(c->window) || c->window == EVA_WINDOW_NONCAUSAL) return EVA_ERR_INVALID;
    if (c->R < 32 || c->R % 32 != 0 || c->S_max < 32 || c->S_max % 32 != 0) return EVA_ERR_INVALID;
    if ((long long)c->R < (long long)c->W + c->C - 1) return EVA_ERR_CAPACITY;
    // summaries are built as chunks complete: up to max_tok / C of them
    if (c->max_tok / c->C > c->S_max) return EVA_ERR_CAPACITY;
    if ((long long)c->B * c->H_kv > 65535) return EVA_ERR_UNSUPPORTED;
    if (c->rf != 0 && c->rf != 1) return EVA_ERR_INVALID;
    if (c->rf && (!(c->rf_lambda >= 0.f) || c->rf_lambda > 1e30f)) return EVA_ERR_INVALID;
    return EVA_OK;
}

eva::CacheView rview_of(const eva_rcache* c) {
    eva::CacheView v;
    v.B = c->B;
    v.H = c->H;
    v.Hkv = c->H_kv;
    v.W = c->W;
    v.C = c->C;
    v.R = c->R;
    v.S_max = c->S_max;
    v.n_tok = 0;  // per-sequence counts live in device memory
    v.window = c->window;
    v.k_ring = c->k_ring;
    v.vt_ring = c->vt_ring;
    v.k_sum = c->k_sum;
    v.vt_sum = c->vt_sum;
    v.rf = c->rf;
    v.rf_scale = rf_scale_of(c->rf, c->rf_lambda, c->d);
    v.rf_seed = c->rf_seed;
    return v;
}

eva::RaggedState rstate_of(const eva_rcache* c, const int* active) {
    return eva::RaggedState{c->n_tok, c->arrive, active, c->max_tok};
}

// Most 32-row chunks a decode row of a ragged cache can touch: the summaries
// of a sequence at max_tok tokens plus a window starting anywhere in a tile.
int rdecode_max_chunks(const eva_rcache* c) {
    int n_sum = prefix_summaries(c->window, c->max_tok - 1, c->W, c->C);
    if (n_sum > c->S_max) n_sum = c->S_max;
    // longest window: W, or W + C - 1 when extended down to its chunk
    long long w = c->window == EVA_WINDOW_CHUNK_ALIGNED ? (long long)c->W + c->C - 1 : c->W;
    const int win = (int)(w < c->max_tok ? w : c->max_tok);
    return (n_sum + 31) / 32 + (win + 30) / 32 + 1;
}

// Index of the chunk whose last token is position p, or -1: its summary is
// built by the step that appends p.
int completed_chunk(long long p, int C) { return (p + 1) % C == 0 ? (int)((p + 1) / C - 1) : -1; }

int decode_chunks(const eva_cache* c, long long p, int* n_sum_out, int* win_lo_out, int* n_sum_chunks,
                  int* n_win_chunks) {
    const int n_sum = prefix_summaries(c->window, p, c->W, c->C);
    const long long win_lo = window_lo(c->window, p, c->W, c->C);
    *n_sum_out = n_sum;
    *win_lo_out = (int)win_lo;
    *n_sum_chunks = (n_sum + 31) / 32;
    *n_win_chunks = (int)(p / 32 - win_lo / 32 + 1);
    return *n_sum_chunks + *n_win_chunks;
}

}  // namespace

extern "C" {

const char* eva_status_string(int status) {
    switch (status) {
        case EVA_OK: return "ok";
        case EVA_ERR_INVALID: return "invalid argument";
        case EVA_ERR_UNSUPPORTED: return "unsupported head dimension, element type or size";
        case EVA_ERR_CAPACITY: return "cache capacity exceeded";
        case EVA_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int eva_build_summaries(const void* K, const void* V, void* Ksum, void* Vsum, int B, int H_kv, int L, int d, int C,
                        int dtype, void* stream) {
    if (B < 1 || H_kv < 1 || L < 1 || C < 1) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    int st = supported(d, dtype);
    if (st != EVA_OK) return st;
    if (C > kMaxChunk) return EVA_ERR_UNSUPPORTED;
    if ((long long)B * H_kv > 65535) return EVA_ERR_UNSUPPORTED;
    if (L / C == 0) return EVA_OK;
    if (!K || !V || !Ksum || !Vsum) return EVA_ERR_INVALID;
    if (!aligned16(K) || !aligned16(V)) return EVA_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(dispatch(d, dtype, [&](auto dd, auto t) {
        return eva::launch_summaries<decltype(dd)::value, decltype(t)>(K, V, Ksum, Vsum, B * H_kv, L, C, nullptr,
                                                                       0.f, s);
    }));
}

int eva_build_summaries_rf(const void* K, const void* V, const float* eps, float lambda, void* Ksum, void* Vsum,
                           int B, int H_kv, int L, int d, int C, int dtype, void* stream) {
    if (B < 1 || H_kv < 1 || L < 1 || C < 1) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (!(lambda >= 0.f) || lambda > 1e30f) return EVA_ERR_INVALID;  // rejects NaN and infinities
    int st = supported(d, dtype);
    if (st != EVA_OK) return st;
    if (C > kMaxChunk) return EVA_ERR_UNSUPPORTED;
    if ((long long)B * H_kv > 65535) return EVA_ERR_UNSUPPORTED;
    if (L / C == 0) return EVA_OK;
    if (!K || !V || !Ksum || !Vsum || !eps) return EVA_ERR_INVALID;
    if (!aligned16(K) || !aligned16(V) || !aligned16(eps)) return EVA_ERR_INVALID;
    const float rf_scale = (float)(lambda * sqrt(sqrt((double)d)));
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(dispatch(d, dtype, [&](auto dd, auto t) {
        return eva::launch_summaries<decltype(dd)::value, decltype(t)>(K, V, Ksum, Vsum, B * H_kv, L, C, eps,
                                                                       rf_scale, s);
    }));
}

int eva_rf_noise(float* eps, int B, int H_kv, int n_chunks, int d, unsigned long long seed, void* stream) {
    if (B < 1 || H_kv < 1 || n_chunks < 0) return EVA_ERR_INVALID;
    if (d != 64 && d != 128) return EVA_ERR_UNSUPPORTED;
    if ((long long)B * H_kv > 65535 || n_chunks > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (n_chunks == 0) return EVA_OK;
    if (!eps || !aligned16(eps)) return EVA_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(d == 64 ? eva::launch_rf_noise<64>(eps, B * H_kv, n_chunks, seed, s)
                              : eva::launch_rf_noise<128>(eps, B * H_kv, n_chunks, seed, s));
}

int eva_prefill_attention(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum, void* O,
                          int B, int H, int H_kv, int L, int d, int W, int C, int dtype, void* stream) {
    return eva_prefill_attention_ex(Q, K, V, Ksum, Vsum, O, B, H, H_kv, L, d, W, C, dtype, EVA_WINDOW_SLIDING,
                                    stream);
}

// Workgroup geometry of the prefill kernel that runs (bf16: pipelined MFMA
// kernel, fp32: two-phase kernel) and its tile count.
struct PrefillTiles {
    int Gt, pos_per_wg, n_pos_tiles;
    long long n_tiles;
};
static PrefillTiles prefill_tiles(int B, int H, int H_kv, int L, int W, int dtype) {
    const int G = H / H_kv;
    const int waves = dtype != EVA_BF16                   ? eva::kPrefillWaves
                      : eva::prefill_mfma_narrow(G, W) ? eva::kMfmaWavesNarrow
                                                       : eva::kMfmaWavesWide;
    const int cols = dtype == EVA_BF16 ? 16 * eva::kMfmaColBlocks : 32;
    PrefillTiles t;
    t.Gt = gcd(G, waves);
    t.pos_per_wg = cols * waves / t.Gt;
    const long long pos_tiles = ((long long)L + t.pos_per_wg - 1) / t.pos_per_wg;  // L near 2^31 must not wrap
    t.n_pos_tiles = (int)pos_tiles;
    t.n_tiles = (long long)B * H_kv * (G / t.Gt) * pos_tiles;
    return t;
}

static int prefill_attention_impl(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                                  void* O, float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C,
                                  int dtype, int window, void* stream);

int eva_prefill_attention_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                             void* O, int B, int H, int H_kv, int L, int d, int W, int C, int dtype, int window,
                             void* stream) {
    return prefill_attention_impl(Q, K, V, Ksum, Vsum, O, nullptr, nullptr, B, H, H_kv, L, d, W, C, dtype, window,
                                  stream);
}

int eva_prefill_forward_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum, void* O,
                           float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                           int window, void* stream) {
    if (!lse) return EVA_ERR_INVALID;
    if (O_lo && (dtype != EVA_BF16 || !aligned16(O_lo))) return EVA_ERR_INVALID;
    return prefill_attention_impl(Q, K, V, Ksum, Vsum, O, lse, O_lo, B, H, H_kv, L, d, W, C, dtype, window, stream);
}

int eva_prefill_forward(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum, void* O,
                        float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                        void* stream) {
    return eva_prefill_forward_ex(Q, K, V, Ksum, Vsum, O, lse, O_lo, B, H, H_kv, L, d, W, C, dtype,
                                  EVA_WINDOW_SLIDING, stream);
}

static int prefill_attention_impl(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                                  void* O, float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C,
                                  int dtype, int window, void* stream) {
    if (B < 1 || H < 1 || H_kv < 1 || L < 1 || W < 1 || C < 1 || H % H_kv != 0) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (!valid_window(window)) return EVA_ERR_INVALID;
    int st = supported(d, dtype);
    if (st != EVA_OK) return st;
    if (!Q || !K || !V || !O) return EVA_ERR_INVALID;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return EVA_ERR_INVALID;
    const int n_chunks = L / C;
    // a row sees summaries only when some chunk lies wholly outside its window
    if (any_summary(window, L, W, C) && (!Ksum || !Vsum || !aligned16(Ksum) || !aligned16(Vsum)))
        return EVA_ERR_INVALID;

    eva::PrefillParams p{};
    p.Q = Q;
    p.K = K;
    p.V = V;
    p.Ks = Ksum;
    p.Vs = Vsum;
    p.O = O;
    p.B = B;
    p.H = H;
    p.Hkv = H_kv;
    p.L = L;
    p.W = W;
    p.C = C;
    p.n_chunks = n_chunks;
    p.G = H / H_kv;
    const PrefillTiles t = prefill_tiles(B, H, H_kv, L, W, dtype);
    if (t.n_tiles > 0x7fffffffLL) return EVA_ERR_UNSUPPORTED;
    p.Gt = t.Gt;
    p.n_hg = p.G / p.Gt;
    p.pos_per_wg = t.pos_per_wg;
    p.n_pos_tiles = t.n_pos_tiles;
    p.n_tiles = (int)t.n_tiles;
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)d));
    p.log2C = (float)log2((double)C);
    p.window = window;
    p.lse = lse;
    p.O_lo = O_lo;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(dispatch(d, dtype, [&](auto dd, auto t) {
        if constexpr (std::is_same<decltype(t), eva::bf16>::value)
            return eva::launch_prefill_mfma<decltype(dd)::value>(p, s);
        else
            return eva::launch_prefill<decltype(dd)::value, decltype(t)>(p, s);
    }));
}

int eva_cache_fill(eva_cache* cache, const void* K, const void* V, const void* Ksum, const void* Vsum, int L,
                   void* stream) {
    int st = check_cache(cache);
    if (st != EVA_OK) return st;
    if (L < 1 || !K || !V || !aligned16(K) || !aligned16(V)) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    const int n_chunks = L / cache->C;
    if (n_chunks > 0 && (!Ksum || !Vsum || !aligned16(Ksum) || !aligned16(Vsum))) return EVA_ERR_INVALID;
    if (cache->S_max < n_chunks) return EVA_ERR_CAPACITY;
    eva::CacheView v = view_of(cache);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const eva::RaggedState none{};
    hipError_t e = dispatch(cache->d, cache->dtype, [&](auto dd, auto t) {
        return eva::launch_cache_fill<decltype(dd)::value, decltype(t)>(v, K, V, Ksum, Vsum, L, nullptr, none, s);
    });
    if (e != hipSuccess) return EVA_ERR_HIP;
    cache->n_tok = L;
    return EVA_OK;
}

int eva_prefill(const void* Q, const void* K, const void* V, void* O, int B, int H, int H_kv, int L, int d, int W,
                int C, int dtype, void* Ksum, void* Vsum, eva_cache* cache, void* stream) {
    return eva_prefill_ex(Q, K, V, O, B, H, H_kv, L, d, W, C, dtype, EVA_WINDOW_SLIDING, Ksum, Vsum, cache, stream);
}

int eva_prefill_ex(const void* Q, const void* K, const void* V, void* O, int B, int H, int H_kv, int L, int d, int W,
                   int C, int dtype, int window, void* Ksum, void* Vsum, eva_cache* cache, void* stream) {
    if (B < 1 || H < 1 || H_kv < 1 || L < 1 || W < 1 || C < 1 || H % H_kv != 0) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (!valid_window(window)) return EVA_ERR_INVALID;
    if (cache && window == EVA_WINDOW_NONCAUSAL) return EVA_ERR_INVALID;  // no causal decode to feed
    int st = supported(d, dtype);
    if (st != EVA_OK) return st;
    if (C > kMaxChunk) return EVA_ERR_UNSUPPORTED;
    if ((long long)B * H_kv > 65535) return EVA_ERR_UNSUPPORTED;
    if (!Q || !K || !V || !O) return EVA_ERR_INVALID;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return EVA_ERR_INVALID;
    const int n_chunks = L / C;
    if (n_chunks > 0 && (!Ksum || !Vsum || !aligned16(Ksum) || !aligned16(Vsum))) return EVA_ERR_INVALID;
    // everything the attention call checks is checked here, so that a cache
    // is never filled for a call that then fails
    if (prefill_tiles(B, H, H_kv, L, W, dtype).n_tiles > 0x7fffffffLL) return EVA_ERR_UNSUPPORTED;
    if (cache) {
        st = check_cache(cache);
        if (st != EVA_OK) return st;
        if (cache->B != B || cache->H != H || cache->H_kv != H_kv || cache->d != d || cache->W != W ||
            cache->C != C || cache->dtype != dtype || cache->window != window)
            return EVA_ERR_INVALID;
        // this call builds deterministic summaries: a cache of stochastic
        // ones is filled by eva_cache_fill from eva_build_summaries_rf
        if (cache->rf) return EVA_ERR_INVALID;
        if (cache->S_max < n_chunks) return EVA_ERR_CAPACITY;
    }
    st = eva_build_summaries(K, V, Ksum, Vsum, B, H_kv, L, d, C, dtype, stream);
    if (st != EVA_OK) return st;
    // the cache fill runs right after the summaries, while the last rows of
    // K and V are still in the caches (measured ~1% of the step faster)
    if (cache) {
        st = eva_cache_fill(cache, K, V, Ksum, Vsum, L, stream);
        if (st != EVA_OK) return st;
    }
    return eva_prefill_attention_ex(Q, K, V, Ksum, Vsum, O, B, H, H_kv, L, d, W, C, dtype, window, stream);
}

int eva_cache_append(eva_cache* cache, const void* k_new, const void* v_new, void* stream) {
    int st = check_cache(cache);
    if (st != EVA_OK) return st;
    if (!k_new || !v_new) return EVA_ERR_INVALID;
    const long long p = cache->n_tok;
    if (p >= 0x7fffffffLL - 64) return EVA_ERR_CAPACITY;
    if (completed_chunk(p, cache->C) >= cache->S_max) return EVA_ERR_CAPACITY;
    eva::CacheView v = view_of(cache);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = dispatch(cache->d, cache->dtype, [&](auto dd, auto t) {
        return eva::launch_cache_append<decltype(dd)::value, decltype(t)>(v, k_new, v_new, (int)p, s);
    });
    if (e != hipSuccess) return EVA_ERR_HIP;
    cache->n_tok = p + 1;
    return EVA_OK;
}

size_t eva_decode_workspace_bytes(const eva_cache* cache) {
    if (check_cache(cache) != EVA_OK) return 0;
    const int G = cache->H / cache->H_kv;
    const int n_hg = (G + 15) / 16;
    int n_sum, win_lo, nsc, nwc;
    // the larger of a decode at n_tok - 1 and a fused append + decode at n_tok
    const int n_chunks = decode_chunks(cache, cache->n_tok, &n_sum, &win_lo, &nsc, &nwc);
    const int units = cache->B * cache->H_kv * n_hg;
    const int splits = decode_splits(units, n_chunks);
    if (splits == 1) return 0;
    return (size_t)units * splits * 16 * (cache->d + 2) * sizeof(float);
}

// Decode (or fused append + decode) of position pos of a uniform cache.
// With `fixed` the split partials go to the library's fixed device array
// instead of ws (which is then unused).
static int uniform_decode(const eva_cache* cache, long long pos, const void* q, void* o, const void* k_new,
                          const void* v_new, void* ws, size_t ws_bytes, void* stream, bool fixed = false) {
    if (pos > 0x7fffffffLL - 64) return EVA_ERR_CAPACITY;
    if (cache->B > (k_new ? 32767 : 65535)) return EVA_ERR_UNSUPPORTED;  // grid z: B (x2 when appending)
    eva::DecodeParams p{};
    p.c = view_of(cache);
    p.q = q;
    p.o = o;
    p.p = (int)pos;
    const int n_chunks = decode_chunks(cache, p.p, &p.n_sum, &p.win_lo, &p.n_sum_chunks, &p.n_win_chunks);
    if (p.n_sum > cache->S_max) return EVA_ERR_CAPACITY;
    p.first_win_chunk = p.win_lo / 32;
    p.G = cache->H / cache->H_kv;
    p.n_hg = (p.G + 15) / 16;
    const int units = cache->B * cache->H_kv * p.n_hg;
    // fp32 caches: one workgroup per (b, kv head, head group), no split partials
    p.splits = cache->dtype == EVA_F32 ? 1 : decode_splits(units, n_chunks);
    const size_t need = (size_t)units * p.splits * 16 * (cache->d + 2) * sizeof(float);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (fixed) {
        p.ws = nullptr;
        if (p.splits > 1) {
            if (need > eva::kDecodeScratchBytes) return EVA_ERR_CAPACITY;
            if (eva::decode_scratch(s, &p.ws) != hipSuccess) return EVA_ERR_HIP;
        }
    } else {
        if (p.splits > 1 && (!ws || ws_bytes < need || !aligned16(ws))) p.splits = 1;
        p.ws = p.splits > 1 ? static_cast<float*>(ws) : nullptr;
    }
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)cache->d));
    p.log2C = (float)log2((double)cache->C);
    p.k_new = k_new;
    p.v_new = v_new;
    hipError_t e;
    if (cache->dtype == EVA_F32) {
        // fused step on an fp32 cache: the append, then a plain decode of the
        // appended position (same results as the one-launch bf16 form)
        if (k_new) {
            e = cache->d == 64 ? eva::launch_cache_append<64, float>(p.c, k_new, v_new, p.p, s)
                               : eva::launch_cache_append<128, float>(p.c, k_new, v_new, p.p, s);
            if (e != hipSuccess) return EVA_ERR_HIP;
            p.k_new = p.v_new = nullptr;
        }
        e = cache->d == 64 ? eva::launch_decode<64, float>(p, s) : eva::launch_decode<128, float>(p, s);
    } else {
        e = cache->d == 64 ? eva::launch_decode<64, bf16>(p, s) : eva::launch_decode<128, bf16>(p, s);
    }
    return hip_status(e);
}

int eva_decode_step(const eva_cache* cache, const void* q, void* o, void* ws, size_t ws_bytes, void* stream) {
    int st = check_cache(cache);
    if (st != EVA_OK) return st;
    if (!q || !o || !aligned16(q)) return EVA_ERR_INVALID;
    if (cache->n_tok < 1) return EVA_ERR_INVALID;
    return uniform_decode(cache, cache->n_tok - 1, q, o, nullptr, nullptr, ws, ws_bytes, stream);
}

static int append_decode(eva_cache* cache, const void* q, const void* k_new, const void* v_new, void* o, void* ws,
                         size_t ws_bytes, void* stream, bool fixed) {
    int st = check_cache(cache);
    if (st != EVA_OK) return st;
    if (!q || !o || !k_new || !v_new || !aligned16(q) || !aligned16(k_new)) return EVA_ERR_INVALID;
    const long long p = cache->n_tok;
    if (completed_chunk(p, cache->C) >= cache->S_max) return EVA_ERR_CAPACITY;
    st = uniform_decode(cache, p, q, o, k_new, v_new, ws, ws_bytes, stream, fixed);
    if (st != EVA_OK) return st;
    cache->n_tok = p + 1;
    return EVA_OK;
}

int eva_append_decode(eva_cache* cache, const void* q, const void* k_new, const void* v_new, void* o, void* ws,
                      size_t ws_bytes, void* stream) {
    return append_decode(cache, q, k_new, v_new, o, ws, ws_bytes, stream, false);
}

int eva_append_decode_noalloc(eva_cache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                              void* stream) {
    return append_decode(cache, q, k_new, v_new, o, nullptr, 0, stream, true);
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------

namespace {
size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }
// fp32 scratch of the backward: row dots, summary gradients, and the
// per-chunk / per-key factors through which the summaries reach dK and dV
struct BwdLayout {
    size_t dv, dksw, dvsw, khat, dkhat, da, bw, total;
};
BwdLayout bwd_layout(long long B, long long H, long long H_kv, long long L, long long d, long long C) {
    BwdLayout l;
    const long long nc = L / C;
    const size_t vec = (size_t)(B * H_kv * nc * d) * 4;
    const size_t key = (size_t)(B * H_kv * nc * C) * 4;
    const size_t split = (size_t)eva::bwd_summary_splits(B, H_kv, L, C, H / H_kv);
    l.dv = 0;
    l.dksw = align256(l.dv + (size_t)(B * H * L) * 4);
    l.dvsw = align256(l.dksw + split * vec);
    l.khat = align256(l.dvsw + split * vec);
    l.dkhat = align256(l.khat + vec);
    l.da = align256(l.dkhat + vec);
    l.bw = align256(l.da + key);
    l.total = align256(l.bw + key);
    return l;
}
}  // namespace

size_t eva_prefill_backward_workspace_bytes(int B, int H, int H_kv, int L, int d, int C) {
    if (B < 1 || H < 1 || H_kv < 1 || L < 1 || C < 1 || d < 1) return 0;
    return bwd_layout(B, H, H_kv, L, d, C).total;
}

int eva_prefill_backward_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                            const void* O, const void* O_lo, const void* dO, const float* lse, void* dQ, void* dK,
                            void* dV, void* ws, size_t ws_bytes, int B, int H, int H_kv, int L, int d, int W, int C,
                            int dtype, int window, void* stream) {
    if (B < 1 || H < 1 || H_kv < 1 || L < 1 || W < 1 || C < 1 || H % H_kv != 0) return EVA_ERR_INVALID;
    if (!valid_window(window)) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    int st = supported(d, dtype);
    if (st != EVA_OK) return st;
    if (dtype != EVA_BF16) return EVA_ERR_UNSUPPORTED;
    if (C > kMaxChunk) return EVA_ERR_UNSUPPORTED;
    // grid sizes of the backward kernels (64-row query and key tiles)
    if ((long long)B * H * ((L + 63) / 64) > 0x7fffffffLL) return EVA_ERR_UNSUPPORTED;
    const void* must[] = {Q, K, V, O, dO, lse, dQ, dK, dV, ws};
    for (const void* ptr : must)
        if (!ptr || !aligned16(ptr)) return EVA_ERR_INVALID;
    if (O_lo && !aligned16(O_lo)) return EVA_ERR_INVALID;
    const int n_chunks = L / C;
    if (n_chunks > 0 && (!Ksum || !Vsum || !aligned16(Ksum) || !aligned16(Vsum))) return EVA_ERR_INVALID;
    const BwdLayout lay = bwd_layout(B, H, H_kv, L, d, C);
    if (ws_bytes < lay.total) return EVA_ERR_CAPACITY;
    char* w = static_cast<char*>(ws);
    eva::BwdParams p{};
    p.Q = Q;
    p.K = K;
    p.V = V;
    p.Ks = Ksum;
    p.Vs = Vsum;
    p.O = O;
    p.O_lo = O_lo;
    p.dO = dO;
    p.lse = lse;
    p.dQ = dQ;
    p.dK = dK;
    p.dV = dV;
    p.Dv = reinterpret_cast<float*>(w + lay.dv);
    p.dKs_w = reinterpret_cast<float*>(w + lay.dksw);
    p.dVs_w = reinterpret_cast<float*>(w + lay.dvsw);
    p.khat_w = reinterpret_cast<float*>(w + lay.khat);
    p.dkhat_w = reinterpret_cast<float*>(w + lay.dkhat);
    p.da_w = reinterpret_cast<float*>(w + lay.da);
    p.bw_w = reinterpret_cast<float*>(w + lay.bw);
    p.B = B;
    p.H = H;
    p.Hkv = H_kv;
    p.L = L;
    p.W = W;
    p.C = C;
    p.n_chunks = n_chunks;
    p.n_split = eva::bwd_summary_splits(B, H_kv, L, C, H / H_kv);
    p.window = window;
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)d));
    p.log2C = (float)log2((double)C);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = d == 64 ? eva::launch_backward<64>(p, s) : eva::launch_backward<128>(p, s);
    return hip_status(e);
}

int eva_prefill_backward(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                         const void* O, const void* O_lo, const void* dO, const float* lse, void* dQ, void* dK, void* dV,
                         void* ws, size_t ws_bytes, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                         void* stream) {
    return eva_prefill_backward_ex(Q, K, V, Ksum, Vsum, O, O_lo, dO, lse, dQ, dK, dV, ws, ws_bytes, B, H, H_kv, L, d,
                                   W, C, dtype, EVA_WINDOW_SLIDING, stream);
}

// ---------------------------------------------------------------------------
// ragged caches
// ---------------------------------------------------------------------------

int eva_rcache_fill(const eva_rcache* cache, const void* K, const void* V, const void* Ksum, const void* Vsum,
                    int L, const int* lens, void* stream) {
    int st = check_rcache(cache);
    if (st != EVA_OK) return st;
    if (L < 1 || !K || !V || !lens) return EVA_ERR_INVALID;
    if (L > kMaxLen) return EVA_ERR_UNSUPPORTED;
    if (!aligned16(K) || !aligned16(V)) return EVA_ERR_INVALID;
    const int n_chunks = L / cache->C;
    if (n_chunks > 0 && (!Ksum || !Vsum || !aligned16(Ksum) || !aligned16(Vsum))) return EVA_ERR_INVALID;
    if (cache->S_max < (L < cache->max_tok ? L : cache->max_tok) / cache->C) return EVA_ERR_CAPACITY;
    eva::CacheView v = rview_of(cache);
    const eva::RaggedState r = rstate_of(cache, nullptr);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(dispatch(cache->d, cache->dtype, [&](auto dd, auto t) {
        return eva::launch_cache_fill<decltype(dd)::value, decltype(t)>(v, K, V, Ksum, Vsum, L, lens, r, s);
    }));
}

int eva_rcache_append(const eva_rcache* cache, const void* k_new, const void* v_new, const int* active,
                      void* stream) {
    int st = check_rcache(cache);
    if (st != EVA_OK) return st;
    if (!k_new || !v_new) return EVA_ERR_INVALID;
    eva::CacheView v = rview_of(cache);
    const eva::RaggedState r = rstate_of(cache, active);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(dispatch(cache->d, cache->dtype, [&](auto dd, auto t) {
        return eva::launch_rcache_append<decltype(dd)::value, decltype(t)>(v, r, k_new, v_new, s);
    }));
}

size_t eva_rdecode_workspace_bytes(const eva_rcache* cache) {
    if (check_rcache(cache) != EVA_OK) return 0;
    const int G = cache->H / cache->H_kv;
    const int n_hg = (G + 15) / 16;
    const int units = cache->B * cache->H_kv * n_hg;
    const int splits = decode_splits(units, rdecode_max_chunks(cache));
    if (splits == 1) return 0;
    return (size_t)units * splits * 16 * (cache->d + 2) * sizeof(float);
}

// Decode (k_new == nullptr) or fused append + decode of every active sequence.
static int ragged_decode(const eva_rcache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                         const int* active, void* ws, size_t ws_bytes, void* stream) {
    if (cache->B > (k_new ? 32767 : 65535)) return EVA_ERR_UNSUPPORTED;  // grid z: B (x2 when appending)
    eva::DecodeParams p{};
    p.c = rview_of(cache);
    p.q = q;
    p.o = o;
    p.G = cache->H / cache->H_kv;
    p.n_hg = (p.G + 15) / 16;
    const int units = cache->B * cache->H_kv * p.n_hg;
    p.splits = cache->dtype == EVA_F32 ? 1 : decode_splits(units, rdecode_max_chunks(cache));
    const size_t need = (size_t)units * p.splits * 16 * (cache->d + 2) * sizeof(float);
    if (p.splits > 1 && (!ws || ws_bytes < need || !aligned16(ws))) p.splits = 1;
    p.ws = p.splits > 1 ? static_cast<float*>(ws) : nullptr;
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)cache->d));
    p.log2C = (float)log2((double)cache->C);
    p.n_tok = cache->n_tok;
    p.active = active;
    p.max_tok = cache->max_tok;
    p.k_new = k_new;
    p.v_new = v_new;
    p.arrive = cache->arrive;
    p.arrivals = p.splits * cache->H_kv * p.n_hg + cache->H_kv;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (cache->dtype == EVA_F32) {
        // fused step on an fp32 cache: the ragged append (which advances
        // n_tok), then a plain decode of each sequence's last position
        if (k_new) {
            const eva::RaggedState r = rstate_of(cache, active);
            e = cache->d == 64 ? eva::launch_rcache_append<64, float>(p.c, r, k_new, v_new, s)
                               : eva::launch_rcache_append<128, float>(p.c, r, k_new, v_new, s);
            if (e != hipSuccess) return EVA_ERR_HIP;
            p.k_new = p.v_new = nullptr;
        }
        e = cache->d == 64 ? eva::launch_decode<64, float>(p, s) : eva::launch_decode<128, float>(p, s);
    } else {
        e = cache->d == 64 ? eva::launch_decode<64, bf16>(p, s) : eva::launch_decode<128, bf16>(p, s);
    }
    return hip_status(e);
}

int eva_rdecode_step(const eva_rcache* cache, const void* q, void* o, const int* active, void* ws,
                     size_t ws_bytes, void* stream) {
    int st = check_rcache(cache);
    if (st != EVA_OK) return st;
    if (!q || !o || !aligned16(q)) return EVA_ERR_INVALID;
    return ragged_decode(cache, q, nullptr, nullptr, o, active, ws, ws_bytes, stream);
}

int eva_rappend_decode(const eva_rcache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                       const int* active, void* ws, size_t ws_bytes, void* stream) {
    int st = check_rcache(cache);
    if (st != EVA_OK) return st;
    if (!q || !o || !k_new || !v_new || !aligned16(q) || !aligned16(k_new)) return EVA_ERR_INVALID;
    return ragged_decode(cache, q, k_new, v_new, o, active, ws, ws_bytes, stream);
}

int eva_generate(const eva_rcache* cache, const void* q, const void* k, const void* v, void* o, int T,
                 const int* active, void* ws, size_t ws_bytes, void* stream) {
    int st = check_rcache(cache);
    if (st != EVA_OK) return st;
    if (T < 1 || !q || !k || !v || !o) return EVA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k)) return EVA_ERR_INVALID;
    const size_t es = cache->dtype == EVA_F32 ? 4 : 2;
    const size_t q_step = (size_t)cache->B * cache->H * cache->d * es;
    const size_t kv_step = (size_t)cache->B * cache->H_kv * cache->d * es;
    const char* qc = static_cast<const char*>(q);
    const char* kc = static_cast<const char*>(k);
    const char* vc = static_cast<const char*>(v);
    char* oc = static_cast<char*>(o);
    for (int t = 0; t < T; ++t) {
        st = ragged_decode(cache, qc + t * q_step, kc + t * kv_step, vc + t * kv_step, oc + t * q_step, active, ws,
                           ws_bytes, stream);
        if (st != EVA_OK) return st;
    }
    return EVA_OK;
}

}  // extern "C"
