// Decode-side kernels: cache fill after a prefill, per-token append (with the
// chunk summary that becomes due), and the bandwidth-bound decode step.
//
// Cache layout (per (b, kv head)): keys row-major by ring slot [R][D], values
// transposed per 8-slot tile [R/8][D][8]; summary keys [S_max][D], summary
// values [S_max/8][D][8].  Position p lives in slot p mod R; R is a multiple
// of 32 so a 32-aligned run of positions is 32 consecutive slots, and its
// keys and values are two contiguous 32*D blocks.
//
// Decode works on 32-row chunks: summary chunks (rows of the summary arrays)
// and window chunks (32-aligned position runs of the ring).  Per chunk a wave
// computes S^T = K Q^T with the matrix cores, reading the key rows straight
// from HBM as A operands (rows permuted so that each lane's 8 softmax weights
// land on 8 consecutive keys), then O^T += V^T P^T with the transposed values
// read straight from HBM as A operands: every byte of K and V is read once,
// 16 B per lane, and never staged through LDS.  Query heads sharing a kv head
// (up to 16) are the MFMA columns, so the keys and values are read once for
// all of them.
#include <mutex>

#include "eva_kernels.hpp"
#include "summary.hpp"

namespace eva {

namespace {

// ---------------------------------------------------------------------------
// cache fill
// ---------------------------------------------------------------------------
// One workgroup moves 32 rows: 32 ring positions (32-aligned, so they occupy
// 32 consecutive slots) or 32 summaries.  Keys are copied row by row; values
// go through LDS so the transposed store writes the rows' four contiguous
// [D][8] tiles instead of scattered elements.
// Source arrays have L rows (K, V) and n_chunks rows (Ks, Vs) per (b, g).
// With `lens` each sequence copies only its own valid prefix: the tiles are
// counted from that sequence's first ring position, and tiles past its
// length do nothing.
template <int D, typename T>
__global__ __launch_bounds__(256) void cache_fill_kernel(CacheView c, const T* __restrict__ K, const T* __restrict__ V,
                                                         const T* __restrict__ Ks, const T* __restrict__ Vs, int L,
                                                         int n_chunks, int ring_tiles, const int* __restrict__ lens,
                                                         RaggedState rs) {
    __shared__ T tile[32][D + 2];
    const size_t bg = blockIdx.y;
    int len = L;
    if (lens) {
        const int b = (int)blockIdx.y / c.Hkv;
        len = min(max(lens[b], 0), min(L, rs.max_tok));
        if (blockIdx.x == 0 && (int)blockIdx.y % c.Hkv == 0 && threadIdx.x == 0) {
            rs.n_tok[b] = len;
            rs.arrive[b] = 0;
        }
    }
    const int first = max(0, len - c.R);
    const bool ring = (int)blockIdx.x < ring_tiles;
    int r0, r1, dst0;  // source rows [r0, r1), destination slot/index of r0
    const T *src_k, *src_v;
    T *dst_k, *dst_vt;
    if (ring) {
        const int p0 = (first / 32 + (int)blockIdx.x) * 32;
        r0 = max(p0, first);
        r1 = min(p0 + 32, len);
        dst0 = r0 % c.R;
        src_k = K + bg * (size_t)L * D;
        src_v = V + bg * (size_t)L * D;
        dst_k = static_cast<T*>(c.k_ring) + bg * (size_t)c.R * D;
        dst_vt = static_cast<T*>(c.vt_ring) + bg * (size_t)c.R * D;
    } else {
        r0 = ((int)blockIdx.x - ring_tiles) * 32;
        r1 = min(r0 + 32, len / c.C);
        dst0 = r0;
        src_k = Ks + bg * (size_t)n_chunks * D;
        src_v = Vs + bg * (size_t)n_chunks * D;
        dst_k = static_cast<T*>(c.k_sum) + bg * (size_t)c.S_max * D;
        dst_vt = static_cast<T*>(c.vt_sum) + bg * (size_t)c.S_max * D;
    }
    const int rows = max(r1 - r0, 0);
    if (rows == 32 && dst0 % 32 == 0) {
        // 32 whole rows of the destination: 16-B row copies of K, and their four
        // [D][8] blocks of transposed V written 16 B (one feature's slots, bf16)
        // at a time, consecutive threads on consecutive features
        constexpr int CH = D * (int)sizeof(T) / 16;  // 16-B chunks per row
        constexpr int EPC = 16 / (int)sizeof(T);     // elements per chunk
        for (int e = threadIdx.x; e < 32 * CH; e += blockDim.x) {
            const int r = e / CH, ch = e % CH;
            const size_t so = (size_t)(r0 + r) * D + ch * EPC;
            *reinterpret_cast<u32x4*>(dst_k + (size_t)(dst0 + r) * D + ch * EPC) =
                *reinterpret_cast<const u32x4*>(src_k + so);
            const u32x4 vv = *reinterpret_cast<const u32x4*>(src_v + so);
            const T* ve = reinterpret_cast<const T*>(&vv);
#pragma unroll
            for (int i = 0; i < EPC; ++i) tile[r][ch * EPC + i] = ve[i];
        }
        __syncthreads();
        T* blk = dst_vt + vt_index<D>(0, dst0);
        for (int e = threadIdx.x; e < D * 32 / EPC; e += blockDim.x) {
            const int d = e % D, r8 = (e / D) * EPC;
            u32x4 w;
            T* we = reinterpret_cast<T*>(&w);
#pragma unroll
            for (int i = 0; i < EPC; ++i) we[i] = tile[r8 + i][d];
            *reinterpret_cast<u32x4*>(blk + vt_index<D>(d, r8)) = w;
        }
        return;
    }
    for (int e = threadIdx.x; e < rows * D; e += blockDim.x) {
        const int r = e / D, d = e % D;
        dst_k[(size_t)(dst0 + r) * D + d] = src_k[(size_t)(r0 + r) * D + d];
        tile[r][d] = src_v[(size_t)(r0 + r) * D + d];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < rows * D; e += blockDim.x) {
        const int d = e / rows, r = e % rows;
        dst_vt[vt_index<D>(d, dst0 + r)] = tile[r][d];
    }
}

// ---------------------------------------------------------------------------
// append
// ---------------------------------------------------------------------------
// A chunk's summary is built in the step that appends the chunk's last token:
// the chunk becomes visible only W steps later (s(n) counts chunks ending at
// or before n - W), so the build is never on the path of the decode that
// runs beside it.  Index of the chunk the token at position p completes, or -1.
__device__ inline int chunk_completed(int p, int C) { return (p + 1) % C == 0 ? (p + 1) / C - 1 : -1; }

// Append the token at position p of (b, g) = row bg: build the summary of the
// chunk it completes (from the ring's other C - 1 rows of that chunk and the
// token itself), then write the token to ring slot p mod R.  The slot holds
// position p - R, which belongs to neither that chunk (R >= C) nor any decode
// window (R >= W), so nothing running concurrently reads it.  Called by a
// whole kSummaryThreads workgroup; smem holds C + summary_red_floats<D>().
template <int D, typename T>
__device__ void append_token(const CacheView& c, size_t bg, int p, const T* __restrict__ kn,
                             const T* __restrict__ vn, float* smem) {
    T* kr = static_cast<T*>(c.k_ring) + bg * (size_t)c.R * D;
    T* vr = static_cast<T*>(c.vt_ring) + bg * (size_t)c.R * D;
    const int s_new = chunk_completed(p, c.C);
    if (s_new >= 0 && s_new < c.S_max) {
        RingChunkPlusNew<D, T> src{{kr, vr, (long long)s_new * c.C, c.R}, kn, vn, c.C - 1};
        float kh[8], vh[8];
        if (c.rf) {
            // this thread's 8 features of the chunk's counter-based draw
            const int cc = threadIdx.x % (D / 8);
            float e[8];
            rf_normals4(c.rf_seed, (uint32_t)(2 * cc), (uint32_t)s_new, (uint32_t)bg, e);
            rf_normals4(c.rf_seed, (uint32_t)(2 * cc + 1), (uint32_t)s_new, (uint32_t)bg, e + 4);
            chunk_summary<D, true>(src, c.C, smem, smem + c.C, kh, vh, RfNoise{e, c.rf_scale});
        } else {
            chunk_summary<D>(src, c.C, smem, smem + c.C, kh, vh);
        }
        const int t = threadIdx.x;
        if (t < D / 8) {
            T* ks = static_cast<T*>(c.k_sum) + bg * (size_t)c.S_max * D;
            T* vs = static_cast<T*>(c.vt_sum) + bg * (size_t)c.S_max * D;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                ks[(size_t)s_new * D + t * 8 + i] = from_f32<T>(kh[i]);
                vs[vt_index<D>(t * 8 + i, s_new)] = from_f32<T>(vh[i]);
            }
        }
    }
    const int slot = p % c.R;
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        kr[(size_t)slot * D + d] = kn[d];
        vr[vt_index<D>(d, slot)] = vn[d];
    }
}

// Uniform cache: one workgroup per (b, kv head), position p from the host.
template <int D, typename T>
__global__ __launch_bounds__(kSummaryThreads) void cache_append_kernel(CacheView c, const T* __restrict__ k_new,
                                                                       const T* __restrict__ v_new, int p) {
    extern __shared__ float smem[];
    const size_t bg = blockIdx.x;
    append_token<D, T>(c, bg, p, k_new + bg * D, v_new + bg * D, smem);
}

// Ragged cache: one workgroup per (b, kv head), position p = n_tok[b] read on
// the device; the last of the sequence's H_kv workgroups advances n_tok[b].
template <int D, typename T>
__global__ __launch_bounds__(kSummaryThreads) void rcache_append_kernel(CacheView c, RaggedState rs,
                                                                        const T* __restrict__ k_new,
                                                                        const T* __restrict__ v_new) {
    extern __shared__ float smem[];
    __shared__ int sh_p;
    const size_t bg = blockIdx.x;
    const int b = (int)blockIdx.x / c.Hkv;
    if (rs.active && rs.active[b] == 0) return;
    if (threadIdx.x == 0) sh_p = rs.n_tok[b];
    __syncthreads();
    const int p = sh_p;
    if (p >= rs.max_tok) return;  // full: every workgroup of the sequence agrees
    append_token<D, T>(c, bg, p, k_new + bg * D, v_new + bg * D, smem);
    // Every workgroup of sequence b read n_tok[b] before arriving, so the
    // last to arrive may advance it; it also re-arms the counter.
    if (threadIdx.x == 0) {
        if (atomicAdd(&rs.arrive[b], 1) == c.Hkv - 1) {
            rs.arrive[b] = 0;
            rs.n_tok[b] = p + 1;
        }
    }
}

// ---------------------------------------------------------------------------
// decode step
// ---------------------------------------------------------------------------
constexpr int kDecWaves = 4;
constexpr float kLazyTau = 8.f;  // log2 units: unscaled weights stay <= 256

// Query position and chunk ranges of one decode row.  fresh: the row's own
// token is being appended in the same launch and is read from the inputs.
struct DecodeGeom {
    int p, n_sum, win_lo, n_sum_chunks, n_win_chunks, first_win_chunk;
    bool fresh;
};

// Geometry of sequence b: from the host-computed fields (uniform cache) or
// from the sequence's own token count n (ragged cache).  A plain decode
// serves position n - 1; a fused append + decode appends position n (unless
// the sequence is full) and serves it.  valid = false when the sequence takes
// no part in this step or has no token to serve.
template <bool RAGGED, bool APPEND>
__device__ inline DecodeGeom decode_geom(const DecodeParams& a, int b, bool& valid) {
    DecodeGeom g{a.p, a.n_sum, a.win_lo, a.n_sum_chunks, a.n_win_chunks, a.first_win_chunk, APPEND};
    valid = true;
    if constexpr (RAGGED) {
        const int n = min(a.n_tok[b], a.max_tok);
        g.fresh = APPEND && n < a.max_tok;
        g.p = g.fresh ? n : n - 1;
        valid = g.p >= 0 && !(a.active && a.active[b] == 0);
        g.win_lo = win_lo_rt(a.c.window, g.p, a.c.W, a.c.C);
        g.n_sum = min(g.win_lo / a.c.C, a.c.S_max);  // chunks wholly before the window
        g.n_sum_chunks = (g.n_sum + 31) / 32;
        g.first_win_chunk = g.win_lo / 32;
        g.n_win_chunks = g.p / 32 - g.first_win_chunk + 1;
    }
    return g;
}

// Ragged fused step: every workgroup of sequence b arrives once after its
// last use of n_tok[b]; the last one re-arms the counter and advances the
// count when a token was appended.
template <bool RAGGED, bool APPEND>
__device__ inline void arrive_and_advance(const DecodeParams& a, int b, const DecodeGeom& geo) {
    if constexpr (RAGGED && APPEND) {
        if (threadIdx.x == 0) {
            if (atomicAdd(&a.arrive[b], 1) == a.arrivals - 1) {
                a.arrive[b] = 0;
                if (geo.fresh) a.n_tok[b] = geo.p + 1;
            }
        }
    }
}

// Decode grid: x = split, y = kv head * head group, z = sequence.  With
// APPEND the z range is doubled: z >= B are the appending workgroups, one
// per (sequence, kv head) at x = 0 and head group 0 (the rest exit at once).
// They come last in dispatch order, so they take the slots the decode
// workgroups leave free instead of pushing decode workgroups into a second
// round.
template <int D, bool RAGGED, bool APPEND>
__global__ __launch_bounds__(256) void decode_kernel(DecodeParams a) {
    typedef bf16 T;
    constexpr int NDC = D / 32;  // 32-feature contraction steps
    constexpr int NDB = D / 16;  // 16-feature output blocks
    __shared__ float red_m[kDecWaves][16];
    __shared__ float red_l[kDecWaves][16];
    __shared__ float red_o[kDecWaves][D][17];

    const int split = blockIdx.x;
    const int kvh = blockIdx.y / a.n_hg;
    const int hg = blockIdx.y % a.n_hg;
    const CacheView& c = a.c;
    const bool appender = APPEND && (int)blockIdx.z >= c.B;
    const int b = appender ? (int)blockIdx.z - c.B : (int)blockIdx.z;
    if (appender && (split != 0 || hg != 0)) return;  // idle: reads nothing, does not arrive
    bool valid;
    const DecodeGeom geo = decode_geom<RAGGED, APPEND>(a, b, valid);
    if (!valid) return;  // uniform across the workgroup
    const T* k_new = static_cast<const T*>(a.k_new) + ((size_t)b * c.Hkv + kvh) * D;
    const T* v_new = static_cast<const T*>(a.v_new) + ((size_t)b * c.Hkv + kvh) * D;
    if constexpr (APPEND) {
        if (appender) {
            extern __shared__ float smem[];
            if (geo.fresh) append_token<D, T>(c, (size_t)b * c.Hkv + kvh, geo.p, k_new, v_new, smem);
            arrive_and_advance<RAGGED, APPEND>(a, b, geo);
            return;
        }
    }
    const size_t bg = (size_t)b * c.Hkv + kvh;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // keeps chunk bookkeeping scalar
    const int g = lane >> 4, c16 = lane & 15;
    const int h0 = kvh * a.G + hg * 16;
    const int ncols = min(16, a.G - hg * 16);

    const T* kring = static_cast<const T*>(c.k_ring) + bg * (size_t)c.R * D;
    const T* vring = static_cast<const T*>(c.vt_ring) + bg * (size_t)c.R * D;
    const T* ksum = static_cast<const T*>(c.k_sum) + bg * (size_t)c.S_max * D;
    const T* vsum = static_cast<const T*>(c.vt_sum) + bg * (size_t)c.S_max * D;

    // query fragments: column c16 = head h0 + c16, features dc*32 + 8g .. +7.
    // Columns past ncols repeat the last head: every column's scores,
    // weights and outputs depend on that column alone, and those outputs are
    // never stored.
    bf16x8 qf[NDC];
    {
        const T* qrow = static_cast<const T*>(a.q) + ((size_t)b * c.H + h0 + min(c16, ncols - 1)) * D;
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc) qf[dc] = *reinterpret_cast<const bf16x8*>(qrow + dc * 32 + g * 8);
    }

    // The appended token (row p) in the fragment layouts below: its key as
    // the A-operand fragment of the lane that holds row p, its value feature
    // db*16 + c16 for the lanes whose 8 keys include row p.
    // (each value half in a 32-bit register of its own: packing pairs would
    // make the wave wait for these loads before its first chunk)
    bf16x8 kn[NDC];
    uint32_t vn[NDB];
    if (APPEND && geo.fresh) {
#pragma unroll
        for (int dc = 0; dc < NDC; ++dc) kn[dc] = *reinterpret_cast<const bf16x8*>(k_new + dc * 32 + g * 8);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
            vn[db] = __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(v_new) + db * 16 + c16);
    }

    floatx4 acc[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db) acc[db] = floatx4{0.f, 0.f, 0.f, 0.f};
    // Running reference max (log2 units, per column) and row sum.  The
    // reference moves only when a chunk's max exceeds it by more than
    // kLazyTau, so most chunks add exp2(s - m_run) <= 2^kLazyTau without
    // rescaling the accumulators; the final division by l_run is exact for
    // any reference.
    float m_run = -INFINITY, l_run = 0.f;

    const int n_chunks = geo.n_sum_chunks + geo.n_win_chunks;
    const int worker = split * kDecWaves + wave;
    const int n_workers = a.splits * kDecWaves;
    // Per-lane element offsets inside a 32-row tile.  A operand of S^T = K Q^T
    // for key block kb: row c16 of the block is key krow0 + 4kb, so the keys
    // of lane group g' = c16/4 land on 8 consecutive keys 8g'..8g'+7.
    // A operand of O^T += V^T P^T: feature db*16 + c16, keys 8g .. 8g+7 (the
    // 16 bytes of that feature in the chunk's value tile g).
    const int krow0 = (c16 >> 2) * 8 + (c16 & 3);
    const int koff = krow0 * D + g * 8;
    const int voff = (int)vt_index<D>(c16, 8 * g);

    for (int ch = worker; ch < n_chunks; ch += n_workers) {
        const bool is_sum = ch < geo.n_sum_chunks;
        const T* kt;  // the chunk's key tile [32][D]
        const T* vt;  // the chunk's values: four [D][8] tiles
        int key_lo, key_hi;  // valid chunk keys: [key_lo, key_hi]
        int chunk_pos0 = 0;  // first position of a window chunk
        if (is_sum) {
            const int r0 = ch * 32;
            kt = ksum + (size_t)r0 * D;
            vt = vsum + (size_t)r0 * D;
            key_lo = 0;
            key_hi = min(31, geo.n_sum - 1 - r0);
        } else {
            const int pos0 = (geo.first_win_chunk + ch - geo.n_sum_chunks) * 32;
            const int slot0 = pos0 % c.R;
            chunk_pos0 = pos0;
            kt = kring + (size_t)slot0 * D;
            vt = vring + (size_t)slot0 * D;
            key_lo = max(0, geo.win_lo - pos0);
            key_hi = min(31, geo.p - pos0);
        }
        const bool full = key_lo == 0 && key_hi == 31;
        const unsigned span = (unsigned)(key_hi - key_lo);

        // all 16-B fragment loads of the chunk before any wait: 2*NDC key + NDB
        // value.  Non-temporal: a step reads each cache row once, and keeping
        // the stream out of the caches measured 8% faster (29.7 -> 27.3 us on
        // 64 sequences x 8 kv heads, 576 rows each).  Buffer loads over the
        // chunk's tiles: a lane whose key row, or whose 8 value slots, lie
        // outside [key_lo, key_hi] gets an offset past the tile and reads
        // zeros without a memory access, so the rows a window edge or the last
        // summary tile does not use are not fetched (no branch, no wait).
        constexpr int kTileBytes = 32 * D * (int)sizeof(T);
        constexpr int kSkip = 0x40000000;  // beyond any tile: zeros, no access
        const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(kt), 0, kTileBytes,
                                                                             0x00020000);
        const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(vt), 0, kTileBytes,
                                                                             0x00020000);
        auto ldb = [](__amdgpu_buffer_rsrc_t r, int byte_off) {
            return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 2));  // nt
        };
        bf16x8 ka[2][NDC], va[NDB];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const bool use = (unsigned)(krow0 + 4 * kb - key_lo) <= span;
            const int base = use ? (koff + kb * 4 * D) * (int)sizeof(T) : kSkip;
#pragma unroll
            for (int dc = 0; dc < NDC; ++dc) ka[kb][dc] = ldb(krs, base + dc * 32 * (int)sizeof(T));
        }
        {
            const bool use = g * 8 <= key_hi && g * 8 + 7 >= key_lo;
            const int base = use ? voff * (int)sizeof(T) : kSkip;
#pragma unroll
            for (int db = 0; db < NDB; ++db) va[db] = ldb(vrs, base + db * 16 * kVtTile * (int)sizeof(T));
        }
        __builtin_amdgcn_sched_barrier(0);
        if (APPEND && geo.fresh && !is_sum && chunk_pos0 + 32 > geo.p) {
            // the chunk holding row p: its ring slot is stale, take the input
            const int kp = geo.p - chunk_pos0;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bool mine = krow0 + 4 * kb == kp;
#pragma unroll
                for (int dc = 0; dc < NDC; ++dc) ka[kb][dc] = mine ? kn[dc] : ka[kb][dc];
            }
            const uint32_t lo_here = (unsigned)(kp - g * 8) < 8u && (kp & 1) == 0 ? 1u : 0u;
            const uint32_t hi_here = (unsigned)(kp - g * 8) < 8u && (kp & 1) == 1 ? 1u : 0u;
            const int word = (kp - g * 8) >> 1;
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
                u32x4 w = __builtin_bit_cast(u32x4, va[db]);
                uint32_t bits = vn[db];
                asm volatile("" : "+v"(bits));  // keeps the shift below out of the loop preheader
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (lo_here && word == i) w[i] = (w[i] & 0xffff0000u) | bits;
                    if (hi_here && word == i) w[i] = (w[i] & 0x0000ffffu) | (bits << 16);
                }
                va[db] = __builtin_bit_cast(bf16x8, w);
            }
        }

        // S^T = K Q^T over the chunk: s[kb] rows = keys 8g + 4kb + i
        floatx4 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int dc = 0; dc < NDC; ++dc) s[kb] = mfma_bf16(ka[kb][dc], qf[dc], s[kb]);
        }
        if (!full) {
            // valid chunk keys are [key_lo, key_hi]: unsigned range test, no branches
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const unsigned rel = (unsigned)(g * 8 + kb * 4 + i - key_lo);
                    s[kb][i] = rel <= span ? s[kb][i] : -INFINITY;
                }
            // stale ring slots may hold any bit pattern: zero their values
            // (keys 8g + 2i and 8g + 2i + 1 share dword i of every fragment)
            uint32_t keep[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const unsigned rel = (unsigned)(g * 8 + 2 * i - key_lo);
                keep[i] = (rel <= span ? 0x0000ffffu : 0u) | (rel + 1 <= span ? 0xffff0000u : 0u);
            }
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
                u32x4 w = __builtin_bit_cast(u32x4, va[db]);
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] &= keep[i];
                va[db] = __builtin_bit_cast(bf16x8, w);
            }
        }
        const float bias = is_sum ? a.log2C : 0.f;
        float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
        mx = xgroup_max(mx) * a.scale_log2 + bias;  // finite: every chunk has a valid key
        const bool raise = mx > m_run + kLazyTau;
        if (__builtin_amdgcn_ballot_w64(raise)) {
            const float m_new = raise ? mx : m_run;
            const float alpha = fast_exp2(m_run - m_new);  // first chunk: exp2(-inf) = 0
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < NDB; ++db) acc[db] *= alpha;
            m_run = m_new;
        }
        const float off = bias - m_run;
        bf16x8 pf;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = fast_exp2(fmaf(s[kb][i], a.scale_log2, off));
                l_run += p;
                pf[kb * 4 + i] = to_bf16(p);
            }

        // O^T += V^T P^T
#pragma unroll
        for (int db = 0; db < NDB; ++db) acc[db] = mfma_bf16(va[db], pf, acc[db]);
    }

    // ---- combine the four waves ----
    const float l_wave = xgroup_sum(l_run);
    if (g == 0) {
        red_m[wave][c16] = m_run;
        red_l[wave][c16] = l_wave;
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) red_o[wave][db * 16 + g * 4 + i][c16] = acc[db][i];
    __syncthreads();

    // thread -> (column, feature run): 16 columns x 16 runs of D/16 features
    const int col = tid & 15;
    const int run = tid >> 4;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, red_m[w][col]);
    float wgt[kDecWaves];
    float lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
        wgt[w] = M == -INFINITY ? 0.f : fast_exp2(red_m[w][col] - M);
        lsum += wgt[w] * red_l[w][col];
    }
    constexpr int FPT = D / 16;  // features per thread
    float out[FPT];
#pragma unroll
    for (int f = 0; f < FPT; ++f) {
        const int d = run * FPT + f;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) v += wgt[w] * red_o[w][d][col];
        out[f] = v;
    }
    arrive_and_advance<RAGGED, APPEND>(a, b, geo);  // thread 0 (column 0) stays to here
    if (col >= ncols) return;
    if (a.splits == 1) {
        const float inv = 1.f / lsum;
        T* orow = static_cast<T*>(a.o) + ((size_t)b * c.H + h0 + col) * D + run * FPT;
#pragma unroll
        for (int f = 0; f < FPT; ++f) orow[f] = to_bf16(out[f] * inv);
    } else {
        // partial: [m, l, o[D]] per (b, kv head, head group, split, column)
        float* w = a.ws + ((((size_t)b * c.Hkv + kvh) * a.n_hg + hg) * a.splits + split) * 16 * (D + 2) +
                   (size_t)col * (D + 2);
        if (run == 0) {
            w[0] = M;
            w[1] = lsum;
        }
#pragma unroll
        for (int f = 0; f < FPT; ++f) w[2 + run * FPT + f] = out[f];
    }
}

// Runs after the decode kernel; for a ragged fused step n_tok[b] has been
// advanced by then, which leaves `valid` (active and serving a token) as the
// decode kernel saw it.
template <int D, bool RAGGED>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeParams a) {
    typedef bf16 T;
    const int kvh = blockIdx.y / a.n_hg;
    const int hg = blockIdx.y % a.n_hg;
    const int b = blockIdx.z;
    const CacheView& c = a.c;
    bool valid;
    decode_geom<RAGGED, false>(a, b, valid);
    if (!valid) return;  // no partials were written for this sequence
    const int ncols = min(16, a.G - hg * 16);
    const float* base = a.ws + (((size_t)b * c.Hkv + kvh) * a.n_hg + hg) * a.splits * 16 * (D + 2);
    for (int e = threadIdx.x; e < ncols * D; e += blockDim.x) {
        const int col = e / D, d = e % D;
        float M = -INFINITY;
        for (int sp = 0; sp < a.splits; ++sp) M = fmaxf(M, base[((size_t)sp * 16 + col) * (D + 2)]);
        float num = 0.f, den = 0.f;
        for (int sp = 0; sp < a.splits; ++sp) {
            const float* w = base + ((size_t)sp * 16 + col) * (D + 2);
            const float wt = w[0] == -INFINITY ? 0.f : fast_exp2(w[0] - M);
            den += wt * w[1];
            num += wt * w[2 + d];
        }
        T* orow = static_cast<T*>(a.o) + ((size_t)b * c.H + kvh * a.G + hg * 16 + col) * D;
        orow[d] = to_bf16(num / den);
    }
}

// fp32 caches: the same decode with fp32 matrix-core products
// (v_mfma_f32_16x16x4_f32), one workgroup per (sequence, kv head, head group
// of 16) and four waves striding over the row's 32-row chunks.  Per lane
// (g, c16), column c16 is query head h0 + c16.  S^T = K Q^T: contraction step
// (j, e) pairs feature 16j + 4g + e of key row c16 (+16 kb) with the same
// feature of the query, so each lane's key operands for four steps are one
// 16-byte load; the result holds keys 16 kb + 4g + i.  O^T += V^T P^T:
// contraction step (kb, i) is key 16 kb + 4g + i, whose weight the lane
// already holds, and whose value of feature 16 db + c16 sits in an 8-slot
// value tile next to the lane's other three keys: again one 16-byte load.
// Slots outside the row's valid range are zeroed before the products (a stale
// ring slot may hold any bit pattern, and 0 * NaN is NaN).
template <int D, bool RAGGED>
__global__ __launch_bounds__(256) void decode_f32_kernel(DecodeParams a) {
    constexpr int NJ = D / 16;  // 16-feature blocks (contraction and output)
    __shared__ float red_m[kDecWaves][16];
    __shared__ float red_l[kDecWaves][16];
    __shared__ float red_o[kDecWaves][D][17];

    const int kvh = blockIdx.y / a.n_hg;
    const int hg = blockIdx.y % a.n_hg;
    const int b = blockIdx.z;
    const CacheView& c = a.c;
    bool valid;
    const DecodeGeom geo = decode_geom<RAGGED, false>(a, b, valid);
    if (!valid) return;  // uniform across the workgroup
    const size_t bg = (size_t)b * c.Hkv + kvh;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const int h0 = kvh * a.G + hg * 16;
    const int ncols = min(16, a.G - hg * 16);

    const float* kring = static_cast<const float*>(c.k_ring) + bg * (size_t)c.R * D;
    const float* vring = static_cast<const float*>(c.vt_ring) + bg * (size_t)c.R * D;
    const float* ksum = static_cast<const float*>(c.k_sum) + bg * (size_t)c.S_max * D;
    const float* vsum = static_cast<const float*>(c.vt_sum) + bg * (size_t)c.S_max * D;

    // query fragments (columns past ncols repeat the last head; their
    // outputs are not stored)
    floatx4 qf[NJ];
    {
        const float* qrow = static_cast<const float*>(a.q) + ((size_t)b * c.H + h0 + min(c16, ncols - 1)) * D;
#pragma unroll
        for (int j = 0; j < NJ; ++j) qf[j] = *reinterpret_cast<const floatx4*>(qrow + 16 * j + 4 * g);
    }
    floatx4 acc[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    const int n_chunks = geo.n_sum_chunks + geo.n_win_chunks;
    for (int ch = wave; ch < n_chunks; ch += kDecWaves) {
        const bool is_sum = ch < geo.n_sum_chunks;
        const float *kt, *vt;  // the chunk's 32 key rows and four [D][8] value tiles
        int key_lo, key_hi;    // valid chunk keys: [key_lo, key_hi]
        if (is_sum) {
            const int r0 = ch * 32;
            kt = ksum + (size_t)r0 * D;
            vt = vsum + (size_t)r0 * D;
            key_lo = 0;
            key_hi = min(31, geo.n_sum - 1 - r0);
        } else {
            const int pos0 = (geo.first_win_chunk + ch - geo.n_sum_chunks) * 32;
            const int slot0 = pos0 % c.R;
            kt = kring + (size_t)slot0 * D;
            vt = vring + (size_t)slot0 * D;
            key_lo = max(0, geo.win_lo - pos0);
            key_hi = min(31, geo.p - pos0);
        }
        const unsigned span = (unsigned)(key_hi - key_lo);
        floatx4 s[2];
        float pw[2][4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = floatx4{0.f, 0.f, 0.f, 0.f};
            const float* krow = kt + (size_t)(16 * kb + c16) * D + 4 * g;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const floatx4 kf = *reinterpret_cast<const floatx4*>(krow + 16 * j);
#pragma unroll
                for (int e = 0; e < 4; ++e) s[kb] = mfma_f32(kf[e], qf[j][e], s[kb]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const unsigned rel = (unsigned)(16 * kb + 4 * g + i - key_lo);
                s[kb][i] = rel <= span ? s[kb][i] : -INFINITY;
            }
        }
        // online softmax in log2 units (the chunk always has a valid key)
        const float bias = is_sum ? a.log2C : 0.f;
        float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
        mx = xgroup_max(mx) * a.scale_log2 + bias;
        if (mx > m_run) {
            const float alpha = fast_exp2(m_run - mx);  // first chunk: exp2(-inf) = 0
            l_run *= alpha;
#pragma unroll
            for (int j = 0; j < NJ; ++j) acc[j] *= alpha;
            m_run = mx;
        }
        const float off = bias - m_run;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pw[kb][i] = fast_exp2(fmaf(s[kb][i], a.scale_log2, off));
                l_run += pw[kb][i];
            }
        // O^T += V^T P^T
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const float* vtile = vt + (size_t)(2 * kb + (g >> 1)) * (kVtTile * D) + 4 * (g & 1);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                floatx4 vf = *reinterpret_cast<const floatx4*>(vtile + (16 * j + c16) * kVtTile);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const unsigned rel = (unsigned)(16 * kb + 4 * g + i - key_lo);
                    vf[i] = rel <= span ? vf[i] : 0.f;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[j] = mfma_f32(vf[i], pw[kb][i], acc[j]);
            }
        }
    }

    // ---- combine the four waves (as in decode_kernel) ----
    const float l_wave = xgroup_sum(l_run);
    if (g == 0) {
        red_m[wave][c16] = m_run;
        red_l[wave][c16] = l_wave;
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) red_o[wave][j * 16 + g * 4 + i][c16] = acc[j][i];
    __syncthreads();
    const int col = tid & 15;
    const int run = tid >> 4;
    if (col >= ncols) return;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, red_m[w][col]);
    float wgt[kDecWaves];
    float lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
        wgt[w] = red_m[w][col] == -INFINITY ? 0.f : fast_exp2(red_m[w][col] - M);
        lsum += wgt[w] * red_l[w][col];
    }
    constexpr int FPT = D / 16;
    const float inv = 1.f / lsum;
    float* orow = static_cast<float*>(a.o) + ((size_t)b * c.H + h0 + col) * D + run * FPT;
#pragma unroll
    for (int f = 0; f < FPT; ++f) {
        const int d = run * FPT + f;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) v += wgt[w] * red_o[w][d][col];
        orow[f] = v * inv;
    }
}

}  // namespace

// ---- scratch of the allocation-free fused decode step ----
// The split partials [m, l, o[D]] of every (b, kv head, head group, split,
// column) of one call, in a fixed array of device memory instead of a
// caller's workspace: each GPU the library runs on holds its own copy until
// the process ends.  Every slot the combine kernel reads is written by the
// same call's decode kernel first, so nothing needs clearing between calls;
// calls that overlap on one GPU share the array and race.
static __device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

hipError_t decode_scratch(hipStream_t stream, float** out) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float* addr[kMaxDevices] = {};
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    int dev = cur;
    if (stream) {
        hipDevice_t sd;
        e = hipStreamGetDevice(stream, &sd);
        if (e != hipSuccess) return e;
        dev = (int)sd;
    }
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        // the array's host-side name is no device address: look the address
        // up once per device, with that device current
        if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (dev != cur) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<float*>(ptr);
    }
    *out = addr[dev];
    return hipSuccess;
}

template <int D, typename T>
hipError_t launch_cache_fill(const CacheView& c, const void* K, const void* V, const void* Ks, const void* Vs,
                             int L, const int* lens, const RaggedState& r, hipStream_t stream) {
    const int n_chunks = L / c.C;
    int ring_tiles;
    if (lens) {
        // any length up to L: min(L, R) positions from an arbitrary start
        // touch at most min(L, R) / 32 + 1 aligned 32-position tiles
        ring_tiles = min(L, c.R) / 32 + 1;
    } else {
        const int first = max(0, L - c.R);
        ring_tiles = (L - 1) / 32 - first / 32 + 1;
    }
    const int sum_tiles = (n_chunks + 31) / 32;
    dim3 grid(ring_tiles + sum_tiles, c.B * c.Hkv);
    hipLaunchKernelGGL((cache_fill_kernel<D, T>), grid, dim3(256), 0, stream, c, static_cast<const T*>(K),
                       static_cast<const T*>(V), static_cast<const T*>(Ks), static_cast<const T*>(Vs), L, n_chunks,
                       ring_tiles, lens, r);
    return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_cache_append(const CacheView& c, const void* k_new, const void* v_new, int p, hipStream_t stream) {
    const size_t lds = (size_t)(c.C + summary_red_floats<D>()) * sizeof(float);
    hipLaunchKernelGGL((cache_append_kernel<D, T>), dim3(c.B * c.Hkv), dim3(kSummaryThreads), lds, stream, c,
                       static_cast<const T*>(k_new), static_cast<const T*>(v_new), p);
    return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_rcache_append(const CacheView& c, const RaggedState& r, const void* k_new, const void* v_new,
                                hipStream_t stream) {
    // any sequence may owe a summary this step
    const size_t lds = (size_t)(c.C + summary_red_floats<D>()) * sizeof(float);
    hipLaunchKernelGGL((rcache_append_kernel<D, T>), dim3(c.B * c.Hkv), dim3(kSummaryThreads), lds, stream, c, r,
                       static_cast<const T*>(k_new), static_cast<const T*>(v_new));
    return hipGetLastError();
}

template <int D, bool RAGGED, bool APPEND>
hipError_t launch_decode_impl(const DecodeParams& p, hipStream_t stream) {
    dim3 grid(p.splits, p.c.Hkv * p.n_hg, p.c.B * (APPEND ? 2 : 1));
    const size_t lds = APPEND ? (size_t)(p.c.C + summary_red_floats<D>()) * sizeof(float) : 0;
    hipLaunchKernelGGL((decode_kernel<D, RAGGED, APPEND>), grid, dim3(256), lds, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.splits == 1) return e;
    hipLaunchKernelGGL((decode_combine_kernel<D, RAGGED>), dim3(1, p.c.Hkv * p.n_hg, p.c.B), dim3(256), 0, stream,
                       p);
    return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_decode(const DecodeParams& p, hipStream_t stream) {
    if constexpr (sizeof(T) == 4) {
        // fp32 caches: plain decode only (the fused calls append first), no splits
        if (p.k_new || p.splits != 1) return hipErrorInvalidValue;
        dim3 grid(1, p.c.Hkv * p.n_hg, p.c.B);
        if (p.n_tok)
            hipLaunchKernelGGL((decode_f32_kernel<D, true>), grid, dim3(256), 0, stream, p);
        else
            hipLaunchKernelGGL((decode_f32_kernel<D, false>), grid, dim3(256), 0, stream, p);
        return hipGetLastError();
    } else {
        if (p.k_new)
            return p.n_tok ? launch_decode_impl<D, true, true>(p, stream)
                           : launch_decode_impl<D, false, true>(p, stream);
        return p.n_tok ? launch_decode_impl<D, true, false>(p, stream) : launch_decode_impl<D, false, false>(p, stream);
    }
}

#define EVA_FILL(D, T)                                                                                      \
    template hipError_t launch_cache_fill<D, T>(const CacheView&, const void*, const void*, const void*, \
                                                const void*, int, const int*, const RaggedState&, hipStream_t);
EVA_FILL(64, bf16)
EVA_FILL(128, bf16)
EVA_FILL(64, float)
EVA_FILL(128, float)
#undef EVA_FILL
#define EVA_RAPPEND(D, T)                                                                                 \
    template hipError_t launch_rcache_append<D, T>(const CacheView&, const RaggedState&, const void*, \
                                                   const void*, hipStream_t);
EVA_RAPPEND(64, bf16)
EVA_RAPPEND(128, bf16)
EVA_RAPPEND(64, float)
EVA_RAPPEND(128, float)
#undef EVA_RAPPEND
template hipError_t launch_cache_append<64, bf16>(const CacheView&, const void*, const void*, int, hipStream_t);
template hipError_t launch_cache_append<128, bf16>(const CacheView&, const void*, const void*, int, hipStream_t);
template hipError_t launch_cache_append<64, float>(const CacheView&, const void*, const void*, int, hipStream_t);
template hipError_t launch_cache_append<128, float>(const CacheView&, const void*, const void*, int, hipStream_t);
template hipError_t launch_decode<64, bf16>(const DecodeParams&, hipStream_t);
template hipError_t launch_decode<128, bf16>(const DecodeParams&, hipStream_t);
template hipError_t launch_decode<64, float>(const DecodeParams&, hipStream_t);
template hipError_t launch_decode<128, float>(const DecodeParams&, hipStream_t);

}  // namespace eva
