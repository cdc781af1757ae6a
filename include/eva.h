/*
 * eva.h — C ABI of the MI355X (gfx950) EVA attention library (libeva.so).
 *
 * EVA attention as FlashEVA computes it (section "FlashEVA": EVA rewritten as
 * one softmax attention over an augmented key/value set; the local set E and
 * the chunk partition P_c come from section "EVA Attention", eq. (eva) and
 * eq. (eva_normalization)):
 *
 *   - the causal sequence is cut into chunks of C tokens, chunk c covering
 *     positions [cC, cC + C);
 *   - each complete chunk becomes one summary pair
 *         khat_c = mean of the chunk's keys
 *         vhat_c = sum_j softmax_j(khat_c . k_j / sqrt(d)) v_j
 *     (query independent: the single-sample property of eq. (eva) lets the
 *     random-feature value be computed once per chunk);
 *   - the query at position n takes ONE softmax over
 *         q_n . k_m / sqrt(d)           for m in [max(0, n-W+1), n]   (window)
 *         q_n . khat_c / sqrt(d) + ln C for c < s(n),
 *                                       s(n) = floor(max(0, n-W+1) / C)
 *     with values v_m and vhat_c.  The + ln C gives each summary the weight
 *     of the C tokens it stands for (eq. (eva_normalization) approximates a
 *     chunk's sum of C exponentials by one).  Tokens between the last
 *     summarized chunk and the window start belong to neither term.
 *
 * Shapes and layouts (all row-major, contiguous, device memory):
 *   Q, O          [B][H][L][d]
 *   K, V          [B][H_kv][L][d]
 *   Ksum, Vsum    [B][H_kv][L / C][d]       (complete chunks only)
 * Grouped-query attention: H must be a multiple of H_kv; query head h reads
 * key/value head h / (H / H_kv).
 *
 * Element types: EVA_BF16 (bfloat16 storage, fp32 accumulation; the softmax
 * weights are rounded to bf16 before the weighted sum of values) or EVA_F32
 * (fp32 throughout).  One call uses one type for every tensor it touches.
 * Head dimension d must be 64 or 128.
 *
 * Streams and ownership: `stream` is a hipStream_t passed as void* (NULL =
 * the default stream).  Every call validates its arguments, enqueues kernels
 * on `stream` and returns; it never allocates, frees or synchronizes.  The
 * caller owns every buffer and must keep it alive until the work completes.
 * Kernel faults surface at the caller's next synchronization.
 *
 * Errors: functions return EVA_OK (0) or a negative eva_status; invalid
 * arguments are rejected before anything is enqueued.  No C++ exception
 * crosses this boundary.
 *
 * Limits: sequence lengths L, a ragged cache's max_tok and a cache's token
 * count stay at or below 2^30 (UNSUPPORTED for a longer L or max_tok;
 * CAPACITY once a cache holds 2^30 tokens), and kernel grids below 2^31
 * workgroups (UNSUPPORTED).
 */
#ifndef EVA_H
#define EVA_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    EVA_OK = 0,
    EVA_ERR_INVALID = -1,     /* bad shape, window, chunk size or null pointer */
    EVA_ERR_UNSUPPORTED = -2, /* head dim, element type or size the library does not handle */
    EVA_ERR_CAPACITY = -3,    /* cache ring or summary array too small */
    EVA_ERR_HIP = -4          /* the HIP runtime refused a launch */
} eva_status;

typedef enum { EVA_BF16 = 0, EVA_F32 = 1 } eva_dtype;

/*
 * Local-window variants (the ablation "EVA Local Window Attention Variants"
 * compares the original EVA's blocked local windows with the sliding window
 * of section "FlashEVA"; that section also names the non-causal form).  Row n
 * attends the exact keys [lo, hi] and the summaries of the complete chunks
 * lying wholly outside them on the side(s) listed:
 *   EVA_WINDOW_SLIDING        lo = max(0, n-W+1), hi = n; chunks before lo.
 *                             The default, and what the functions without
 *                             a window argument compute.
 *   EVA_WINDOW_CHUNK_ALIGNED  the sliding start moved down to the start of
 *                             its chunk: lo = s(n) C with s(n) as above, so
 *                             no token falls between summaries and window.
 *   EVA_WINDOW_BLOCKED        lo = floor(n/W) W, hi = n; chunks before lo.
 *   EVA_WINDOW_NONCAUSAL      the whole block: lo = floor(n/W) W,
 *                             hi = min(L, lo+W) - 1; chunks before lo and
 *                             after hi.  Prefill only (no decode cache).
 */
typedef enum {
    EVA_WINDOW_SLIDING = 0,
    EVA_WINDOW_CHUNK_ALIGNED = 1,
    EVA_WINDOW_BLOCKED = 2,
    EVA_WINDOW_NONCAUSAL = 3
} eva_window;

/*
 * Decode cache: the state one decoded token needs — the exact keys/values of
 * the window and the chunk summaries.  The paper's cache of compressed past
 * context (sections "Introduction" and "Conclusion"; section "Related Work":
 * chunks of tokens summarized into single tokens inside the attention
 * itself): it grows by one summary per C tokens, plus a fixed window.
 * Generation reads it once per token, so decode is bound by memory bandwidth
 * (section "Inference throughput and Memory usage"); the layout below is
 * chosen for that read.
 *
 * The struct is caller-owned host memory; the four arrays are caller-owned
 * device memory of the cache's dtype.  Position p of (b, g) lives in ring slot
 * p mod R.  Values are stored transposed (feature-major) in tiles of 8 slots
 * so the decode kernel can feed them to the matrix cores straight from HBM
 * (each feature's 8 slots are one 16-byte operand fragment), 32 aligned slots'
 * keys and values being two contiguous blocks; appending one token's values
 * touches d / 8 cache lines of 128 bytes:
 *   k_ring   [B][H_kv][R][d]           keys, row per slot
 *   vt_ring  [B][H_kv][R/8][d][8]      values: slot s, feature f at
 *                                      [s/8][f][s%8]
 *   k_sum    [B][H_kv][S_max][d]       summary keys
 *   vt_sum   [B][H_kv][S_max/8][d][8]  summary values, tiled the same way
 * Requirements: R >= W + C - 1 and R a multiple of 32; S_max a multiple of 32.
 * n_tok counts the tokens the cache has absorbed (the same for every
 * sequence of the batch); the library updates it.  `window` is the causal
 * window variant the cache serves (any eva_window but EVA_WINDOW_NONCAUSAL).
 * With rf = 1 the summaries are the paper's stochastic single-sample ones
 * throughout: the caller fills the cache (eva_cache_fill) with summaries
 * from eva_build_summaries_rf(eps = eva_rf_noise(rf_seed), rf_lambda), and
 * every chunk an append completes gets its summary from the same estimator
 * and the same counter-based draw (eva_rf_noise's, for that chunk), so the
 * cache holds what eva_build_summaries_rf over the whole sequence would.
 * rf must be 0 or 1 and rf_lambda finite and >= 0 (INVALID otherwise).
 */
typedef struct eva_cache {
    int B, H, H_kv, d, W, C;
    int dtype;        /* eva_dtype */
    int window;       /* eva_window, causal */
    int R;            /* ring slots per (b, kv head) */
    int S_max;        /* summary capacity per (b, kv head) */
    long long n_tok;  /* tokens held; host-side state */
    void* k_ring;
    void* vt_ring;
    void* k_sum;
    void* vt_sum;
    int rf;           /* summaries of chunks completed by appends: 0 the
                         deterministic ones (eva_build_summaries), 1 the
                         stochastic ones (eva_build_summaries_rf) with the
                         noise eva_rf_noise draws for that chunk */
    float rf_lambda;  /* lambda of the stochastic summaries (rf = 1) */
    unsigned long long rf_seed; /* seed of their noise (rf = 1) */
} eva_cache;

/*
 * Chunk summaries (section "EVA Attention", the single-sample property after
 * eq. (eva_normalization)): for every (b, g) and complete chunk c < L / C,
 *   Ksum[b][g][c] = mean of K[b][g][cC .. cC+C-1]
 *   Vsum[b][g][c] = sum_j softmax_j(Ksum . K_j / sqrt(d)) V_j
 * computed in fp32 and stored in `dtype`.  L < C is valid and writes nothing.
 * Errors: INVALID for null pointers with L >= C, B/H_kv/L/C < 1;
 * UNSUPPORTED for d not in {64, 128} or an unknown dtype.
 */
int eva_build_summaries(const void* K, const void* V, void* Ksum, void* Vsum,
                        int B, int H_kv, int L, int d, int C, int dtype, void* stream);

/*
 * Stochastic random-feature chunk summaries: the paper's single-sample
 * estimator (section "EVA Attention", S = 1; feature map
 * xi(x, w) = exp(w . x - |x|^2 / 2) of section "Random Feature Attention").
 * With one sample per chunk every query-dependent factor cancels and the
 * chunk value is sum_j xi(x_j, w) V_j / sum_j xi(x_j, w) over the chunk's
 * scaled keys x_j = K_j / d^(1/4) (the scaling under which
 * exp(q . k / sqrt(d)) = exp(q' . k')).  The sample is
 *     w = mean_j x_j + lambda * clip(eps_c, -1, 1)
 * (the clipped, downscaled proposal of the ablation "Impact of random feature
 * sampling distribution"; the paper uses lambda = 0.1).  Ksum is the mean
 * key, as in eva_build_summaries; lambda = 0 with keys of equal norm inside
 * each chunk gives eva_build_summaries' result.
 *   eps  device fp32 [B][H_kv][L / C][d], 16-byte aligned: the standard
 *        normal draws, one vector per chunk, supplied by the caller.
 * The prefill kernel takes these summaries as it takes any
 * (eva_prefill_attention).  With eps from eva_rf_noise, a decode cache with
 * rf = 1 and the same seed and lambda builds the chunks its appends complete
 * the same way, with the same draws.
 * Errors: as eva_build_summaries; INVALID for a null or misaligned eps or a
 * negative, NaN or infinite lambda.
 */
int eva_build_summaries_rf(const void* K, const void* V, const float* eps, float lambda, void* Ksum, void* Vsum,
                           int B, int H_kv, int L, int d, int C, int dtype, void* stream);

/*
 * Counter-based noise for the stochastic summaries: eps [B][H_kv][n_chunks][d]
 * (fp32, device, 16-byte aligned) receives standard normal draws, the draw
 * of chunk c of (b, g) depending only on (seed, b * H_kv + g, c): features
 * 4i .. 4i+3 come from one Philox4x32-10 block (Salmon et al., SC 2011;
 * counter (i, c, b * H_kv + g, 0), key = the seed's low and high words), each
 * word pair (x, y) giving two normals by the Box-Muller transform on the
 * 24-bit uniforms u = ((x >> 8) + 1/2) 2^-24, v = ((y >> 8) + 1/2) 2^-24:
 * sqrt(-2 ln u) cos(2 pi v) and sqrt(-2 ln u) sin(2 pi v).  The decode cache
 * draws the same noise for the chunks its appends complete (rf = 1).
 * Errors: INVALID (B, H_kv < 1, n_chunks < 0, null or misaligned eps),
 * UNSUPPORTED (d not 64 or 128, sizes).
 */
int eva_rf_noise(float* eps, int B, int H_kv, int n_chunks, int d, unsigned long long seed, void* stream);

/*
 * EVA prefill (section "FlashEVA"): O = one softmax per row over the window
 * keys and the visible chunk summaries, as described at the top of this file.
 * Builds the summaries first (into Ksum/Vsum, caller-provided, shape
 * [B][H_kv][L / C][d]; may be NULL only when L < C), then runs the fused
 * window + summary attention kernel.  If `cache` is not NULL it must describe
 * the same B, H, H_kv, d, W, C and dtype with S_max >= L / C; the call then
 * also writes the last min(L, R) keys/values into the ring, all L / C
 * summaries into the cache, and sets cache->n_tok = L.  (A cache with rf = 1
 * is INVALID here: this call builds deterministic summaries.)
 * Errors: INVALID (shapes, W < 1, C < 1, H % H_kv != 0, null pointers,
 * cache mismatch), CAPACITY (cache too small), UNSUPPORTED (d, dtype).
 */
int eva_prefill(const void* Q, const void* K, const void* V, void* O,
                int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                void* Ksum, void* Vsum, eva_cache* cache, void* stream);

/*
 * The fused window + summary attention kernel alone (section "FlashEVA"),
 * given summaries already built by eva_build_summaries for the same K, V, C:
 * Ksum, Vsum [B][H_kv][L / C][d].  eva_prefill = eva_build_summaries +
 * eva_prefill_attention (+ eva_cache_fill).  Summary pointers may be NULL
 * when no row sees a summary (L - W < C).
 * Errors: as eva_prefill (no cache).
 */
int eva_prefill_attention(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                          void* O, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                          void* stream);

/*
 * eva_prefill_attention and eva_prefill with a window variant (eva_window).
 * A cache passed to eva_prefill_ex must carry the same window; the
 * non-causal variant takes none.
 * Errors: as the functions without the argument; INVALID for an unknown
 * window or a cache with the non-causal variant or another window.
 */
int eva_prefill_attention_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                             void* O, int B, int H, int H_kv, int L, int d, int W, int C, int dtype, int window,
                             void* stream);
int eva_prefill_ex(const void* Q, const void* K, const void* V, void* O, int B, int H, int H_kv, int L, int d,
                   int W, int C, int dtype, int window, void* Ksum, void* Vsum, eva_cache* cache, void* stream);

/*
 * Training forward: eva_prefill_attention (sliding window) that also stores,
 * for every row, lse[b][h][n] = natural log of the sum of exp(logits) over
 * the row's window keys and summaries (logits q.k / sqrt(d), + ln C for a
 * summary), fp32 [B][H][L], as eva_prefill_backward needs it.
 * O_lo (optional, EVA_BF16 only, NULL to skip): [B][H][L][d] receives the
 * rounding residual of the bf16 output, bf16(o - bf16(o)) for the fp32 row o,
 * so that O + O_lo holds o to about 16 bits.  Passed to eva_prefill_backward
 * it makes the row dots D = dO . o exact to that precision; without it D is
 * taken from the bf16 O, whose rounding moves each gradient row by up to
 * ~2^-8 |dO| |O| |k| / sqrt(d) whatever the row's own magnitude.
 * Errors: as eva_prefill_attention; INVALID for a null lse, or an O_lo that
 * is misaligned or given with EVA_F32.
 */
int eva_prefill_forward(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum, void* O,
                        float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                        void* stream);

/* eva_prefill_forward under a window variant (eva_window), for the backward
 * of the same variant.  Errors: as eva_prefill_forward; INVALID for an
 * unknown window. */
int eva_prefill_forward_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum, void* O,
                           float* lse, void* O_lo, int B, int H, int H_kv, int L, int d, int W, int C, int dtype,
                           int window, void* stream);

/*
 * Backward of the EVA prefill (sliding window, bf16; eva_prefill_backward_ex
 * takes the other window variants): given dO [B][H][L][d],
 * the gradient of a loss with respect to O, writes dQ [B][H][L][d] and
 * dK, dV [B][H_kv][L][d] of that loss — through the window keys and values,
 * the summary keys and values, and the summaries' own dependence on K and V
 * (the mean key, and the softmax(mean . k / sqrt(d))-weighted value; the
 * ln C offset is a constant).  Inputs: the forward's Q, K, V, its summaries
 * Ksum, Vsum [B][H_kv][L / C][d] (eva_build_summaries), its output O and lse
 * (eva_prefill_forward), and optionally its output residual O_lo (NULL: the
 * row dots D = dO . O use the bf16 O alone).  The softmax is recomputed from lse, so nothing of
 * size L x L is stored (FlashAttention-style, section "FlashAttention").
 * ws: caller-owned device scratch of eva_prefill_backward_workspace_bytes()
 * bytes (fp32 row dots, summary gradients, and per-chunk and per-key factors
 * of the summaries' own gradient); every byte the call reads it writes first.
 * Errors: INVALID (shapes, null or misaligned pointers), UNSUPPORTED (dtype
 * other than EVA_BF16, d not 64 or 128), CAPACITY (workspace too small).
 */
int eva_prefill_backward(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                         const void* O, const void* O_lo, const void* dO, const float* lse, void* dQ, void* dK,
                         void* dV, void* ws, size_t ws_bytes, int B, int H, int H_kv, int L, int d, int W, int C,
                         int dtype, void* stream);

/*
 * eva_prefill_backward under a window variant (eva_window; the ablation
 * "EVA Local Window Attention Variants" trains with blocked local windows as
 * well as sliding ones): the gradients of the attention whose row n attends
 * the exact keys [lo(n), hi(n)] and the summaries of the chunks wholly
 * outside them (before, and for EVA_WINDOW_NONCAUSAL after), given the
 * forward of the same variant (eva_prefill_forward_ex).
 * Errors: as eva_prefill_backward; INVALID for an unknown window.
 */
int eva_prefill_backward_ex(const void* Q, const void* K, const void* V, const void* Ksum, const void* Vsum,
                            const void* O, const void* O_lo, const void* dO, const float* lse, void* dQ, void* dK,
                            void* dV, void* ws, size_t ws_bytes, int B, int H, int H_kv, int L, int d, int W, int C,
                            int dtype, int window, void* stream);

/* Workspace eva_prefill_backward needs (0 for invalid sizes). */
size_t eva_prefill_backward_workspace_bytes(int B, int H, int H_kv, int L, int d, int C);

/*
 * Load a decode cache from a prefilled sequence of L tokens (the prompt of a
 * generation, section "Experimental setup" / "Inference throughput and Memory
 * usage"; what the cache holds is the window and summary set of section
 * "FlashEVA" for the next position): the last
 * min(L, R) keys/values go to ring slots p mod R and the L / C summaries
 * (as built by eva_build_summaries) to the summary arrays; n_tok becomes L.
 * K, V [H_kv][L][d] per batch row as in eva_prefill; all four device
 * pointers 16-byte aligned.
 * Errors: INVALID (malformed cache, null or misaligned pointers), CAPACITY
 * (S_max < L / C).
 */
int eva_cache_fill(eva_cache* cache, const void* K, const void* V, const void* Ksum, const void* Vsum,
                   int L, void* stream);

/*
 * Append one token per sequence (autoregressive generation, section
 * "Inference throughput and Memory usage"; the summary it may complete is
 * the chunk summary of section "EVA Attention", as in eva_build_summaries):
 * k_new, v_new [B][H_kv][d].  The token takes position p = cache->n_tok.  If it is the last token of chunk
 * S = (p + 1) / C - 1 (p + 1 a multiple of C), that chunk's summary is built
 * from the chunk's other C - 1 rows in the ring and the token itself; the
 * token is written to slot p mod R and n_tok becomes p + 1.  (A chunk is
 * complete W steps before any query sees it, so building it at completion
 * keeps it off the path of the decode steps in between.)
 * Errors: INVALID (null pointers, malformed cache), CAPACITY (S >= S_max).
 */
int eva_cache_append(eva_cache* cache, const void* k_new, const void* v_new, void* stream);

/*
 * One decode step (section "FlashEVA": the softmax over the window keys and
 * the visible summaries, for a single query; section "Inference throughput
 * and Memory usage": one such step per generated token): q [B][H][d] is the
 * query of position p = n_tok - 1 (the token appended last); o [B][H][d]
 * receives its EVA attention output over the ring window [p-W+1, p] and the
 * summaries c < s(p).  Row p of the prefill of the same tokens gives the same
 * result up to rounding order.
 * `ws` is optional device scratch of `ws_bytes` bytes: with at least
 * eva_decode_workspace_bytes(cache) bytes the rows of each sequence are split
 * over more workgroups (for small B * H_kv); with less (or NULL) the call
 * still works, one workgroup per (b, kv head, 16 query heads).
 * Both cache dtypes decode: bf16 caches with bf16 matrix-core products and
 * fp32 accumulation, fp32 caches with fp32 products (their own kernel, no
 * row splits: `ws` is not used).
 * Errors: INVALID (n_tok == 0, null pointers, malformed cache).
 */
int eva_decode_step(const eva_cache* cache, const void* q, void* o,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * Fused per-token step of generation (section "Inference throughput and
 * Memory usage"): eva_cache_append(k_new, v_new) followed by
 * eva_decode_step(q) in one launch, with the same results (the decoded row
 * reads the new token from k_new, v_new while another workgroup writes it to
 * the ring; the summary the token completes is built beside the decode).
 * (On an EVA_F32 cache the append and the decode are two launches.)
 * Errors: as eva_cache_append and eva_decode_step.
 */
int eva_append_decode(eva_cache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                      void* ws, size_t ws_bytes, void* stream);

/* Workspace that lets eva_decode_step / eva_append_decode split rows across
 * workgroups (sized for the next position, n_tok). */
size_t eva_decode_workspace_bytes(const eva_cache* cache);

/*
 * eva_append_decode for callers that cannot allocate (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): no workspace
 * argument.  When the rows are split over workgroups, the partial results go
 * to a fixed array of 6.25 MiB (6553600 bytes) of device memory inside the
 * library, one copy per GPU, held until the process ends; its device
 * address is looked up on the first call on each GPU (the device of
 * `stream`).  The call allocates nothing.  Every slot a call reads is
 * written earlier in the same call, so no state carries over; but calls
 * that overlap on one GPU (concurrent streams, or threads) share the array
 * and race: serialize them.  Results are those of eva_append_decode with a
 * workspace of eva_decode_workspace_bytes(cache) bytes.
 * Errors: as eva_append_decode; CAPACITY if the partials exceed the fixed
 * array (they never do for the shapes this library accepts: at most
 * 766 * 16 * (d + 2) floats); HIP if the array's address cannot be found.
 */
int eva_append_decode_noalloc(eva_cache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                              void* stream);

/*
 * Ragged decode cache: batched generation where every sequence of the batch
 * holds its own number of tokens (section "Inference throughput and Memory
 * usage": many sequences generated in parallel after a prompt; prompts of
 * different lengths make the batch ragged).  The arrays and their layouts are
 * those of eva_cache; what differs is that the token counts live in device
 * memory and are read and advanced by the kernels themselves, so a generation
 * step carries no host-side state and a captured graph of it can be replayed.
 *   n_tok    device int32 [B]: tokens held by sequence b (set by
 *            eva_rcache_fill, advanced by eva_rcache_append)
 *   arrive   device int32 [B]: the library's per-sequence arrival counters;
 *            the caller zeroes them once, every call leaves them zero
 *   max_tok  host: the most tokens any sequence may hold.  S_max must hold
 *            the summaries of every chunk such a sequence completes
 *            (S_max >= max_tok / C).  A sequence that is full ignores
 *            further appends (its n_tok stays max_tok).
 * Sequence b's position p lives in ring slot p mod R of row (b, kv head),
 * exactly as in eva_cache.  Requirements on R and S_max as for eva_cache.
 */
typedef struct eva_rcache {
    int B, H, H_kv, d, W, C;
    int dtype;        /* eva_dtype */
    int window;       /* eva_window, causal */
    int R;
    int S_max;
    int max_tok;
    int* n_tok;
    int* arrive;
    void* k_ring;
    void* vt_ring;
    void* k_sum;
    void* vt_sum;
    int rf;           /* as in eva_cache */
    float rf_lambda;
    unsigned long long rf_seed;
} eva_rcache;

/*
 * Load a ragged cache from a right-padded prefill: K, V [B][H_kv][L][d] and
 * their summaries Ksum, Vsum [B][H_kv][L / C][d] (eva_build_summaries over
 * the padded batch; causality makes every row and every complete chunk below
 * a sequence's own length independent of the padding).  lens is device int32
 * [B], the valid length of each sequence; a length is clamped to
 * [0, min(L, max_tok)].  For each b the last min(len, R) positions go to the
 * ring, summaries c < len / C to the summary arrays, and n_tok[b] = len.
 * K, V, Ksum, Vsum 16-byte aligned.
 * Errors: INVALID (malformed cache, null or misaligned pointers, L < 1),
 * CAPACITY (S_max < min(L, max_tok) / C).
 */
int eva_rcache_fill(const eva_rcache* cache, const void* K, const void* V, const void* Ksum, const void* Vsum,
                    int L, const int* lens, void* stream);

/*
 * Append one token to every active sequence: k_new, v_new [B][H_kv][d].
 * Sequence b's token takes position p = n_tok[b]; if it completes a chunk,
 * that chunk's summary is built (as in eva_cache_append), the token is
 * written and n_tok[b] becomes p + 1.
 * `active` is device int32 [B] (nonzero = append) or NULL for all; inactive
 * and full sequences are left unchanged.
 * Errors: INVALID (malformed cache, null pointers).
 */
int eva_rcache_append(const eva_rcache* cache, const void* k_new, const void* v_new, const int* active,
                      void* stream);

/*
 * One decode step of every active sequence: q [B][H][d] holds, for each b,
 * the query of position n_tok[b] - 1 (its token appended last); o [B][H][d]
 * receives the EVA attention output over that sequence's window and visible
 * summaries, the result of eva_decode_step for a cache holding n_tok[b]
 * tokens.  Rows of inactive sequences and of sequences holding no token are
 * not written.  `ws` as in eva_decode_step, sized by
 * eva_rdecode_workspace_bytes (splits are chosen for the longest sequence a
 * cache of max_tok tokens may hold).
 * fp32 caches decode with their own kernel (no row splits).
 * Errors: INVALID (malformed cache, null pointers).
 */
int eva_rdecode_step(const eva_rcache* cache, const void* q, void* o, const int* active, void* ws,
                     size_t ws_bytes, void* stream);

/*
 * Fused generation step of every active sequence: eva_rcache_append(k_new,
 * v_new, active) followed by eva_rdecode_step(q, active) in one launch, with
 * the same results.  A full sequence appends nothing and decodes its last
 * position, as the two separate calls would.
 * Errors: as eva_rcache_append and eva_rdecode_step.
 */
int eva_rappend_decode(const eva_rcache* cache, const void* q, const void* k_new, const void* v_new, void* o,
                       const int* active, void* ws, size_t ws_bytes, void* stream);

/* Workspace that lets eva_rdecode_step / eva_rappend_decode split rows across
 * workgroups. */
size_t eva_rdecode_workspace_bytes(const eva_rcache* cache);

/*
 * T generation steps (section "Inference throughput and Memory usage"): for
 * t = 0 .. T-1, append token t of every active sequence and decode it.
 *   q, o  [T][B][H][d];  k, v  [T][B][H_kv][d]
 * Equivalent to T calls of eva_rappend_decode(q[t], k[t], v[t]) -> o[t]
 * (one launch per step, two when rows are split over workgroups); all
 * launches are enqueued on `stream` before the call returns (the caller may
 * capture them into a graph).
 * Errors: as eva_rcache_append and eva_rdecode_step; INVALID for T < 1.
 */
int eva_generate(const eva_rcache* cache, const void* q, const void* k, const void* v, void* o, int T,
                 const int* active, void* ws, size_t ws_bytes, void* stream);

/* Static description of an eva_status value. */
const char* eva_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* EVA_H */
