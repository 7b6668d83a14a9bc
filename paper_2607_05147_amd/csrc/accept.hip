// Speculative acceptance over the vocabulary on gfx950 (the left-to-right
// acceptance rule of the speculative-decoding background section).
//
// The vocabulary is cut into 4096-entry chunks.  Kernels, in stream order:
//   rowpass  one pass over every verified logit row: per (row, chunk) the max
//            and argmax of the raw logits (greedy) or the max and the sum of
//            exp2 of the scaled logits (stochastic).  Each wave is an
//            independent persistent worker that streams chunks with the next
//            chunk's loads in flight while it reduces the current one; there
//            are no workgroup barriers.
//   resolve  one workgroup per request: row statistics from the chunk
//            statistics, the accept test of every draft (greedy match or
//            u < p_t(x) / p_d(x)), the first rejection, and what to draw from.
//   resid    stochastic requests with a rejection: one wave per chunk, the
//            mass of the residual max(0, p_t - p_d) of the rejected row.
//   draw     one workgroup per stochastic request: inverse CDF at u[r, K] over
//            the chunk masses, then inside the selected chunk only.
//   rate     (optional) sum_v min(p_t, p_d) per tested row, one wave per chunk,
//            then summed per row.
// Probabilities are evaluated in fp32 (exp2 of log2e-scaled logits); masses
// are accumulated in fp64 across lanes and chunks.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace dspark {

constexpr int kChunk = 4096;                   // vocabulary entries per chunk
constexpr int kLanes = DSPARK_WAVE;
constexpr int kBlk = 256;                      // threads per workgroup
constexpr int kWaves = kBlk / kLanes;
constexpr int kLanePer = kChunk / kLanes;      // 64 entries per lane and chunk
constexpr int kThreadPer = kChunk / kBlk;      // 16 entries per thread (draw)
constexpr int kMaxChunks = 256;                // V <= 2^20
static_assert(kMaxChunks <= kBlk, "the draw loads one chunk mass per thread");
constexpr float kLog2e = 1.4426950408889634f;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct ChunkStat {
    float a;   // greedy: max raw logit      stochastic: max of scaled logit (log2 units)
    float b;   // greedy: unused             stochastic: sum exp2(y - a)
    int arg;   // greedy: argmax (lowest index on ties)
    int pad;
};

struct RowInfo {     // per verified row, written by resolve (stochastic)
    float M, S;      // row max (log2 units) and sum of exp2(y - M)
    int req, t;      // owning request and verify slot
};

struct DrawInfo {    // per request
    int kind;        // 0 none, 1 target row, 2 residual of a rejected row
    int row;         // flattened logit row
    int t;           // verify slot of that row
    int pad;
    float M, S;      // that row's statistics
    int pad2[2];
};

__host__ __device__ static inline int n_chunks(int V) { return (V + kChunk - 1) / kChunk; }

// rows past R*(K+1) do not exist in the workspace: a malformed cu_q is clamped
__device__ __forceinline__ int clamp_rows(int total, int max_rows) {
    return total < 0 ? 0 : (total > max_rows ? max_rows : total);
}

struct AccWs {
    ChunkStat* stats;   // [R*(K+1)][nch]
    RowInfo* rows;      // [R*(K+1)]
    DrawInfo* draw;     // [R]
    double* mass;       // [R][nch]
    double* rate;       // [R*(K+1)][nch]
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static AccWs carve(void* ws, int R, int K, int V) {
    const size_t rows = (size_t)R * (K + 1);
    const int nch = n_chunks(V);
    char* p = (char*)ws;
    AccWs w;
    w.stats = (ChunkStat*)p; p += align256(rows * nch * sizeof(ChunkStat));
    w.rows = (RowInfo*)p;    p += align256(rows * sizeof(RowInfo));
    w.draw = (DrawInfo*)p;   p += align256((size_t)R * sizeof(DrawInfo));
    w.mass = (double*)p;     p += align256((size_t)R * nch * sizeof(double));
    w.rate = (double*)p;
    return w;
}

size_t accept_workspace(int R, int K, int V) {
    const size_t rows = (size_t)R * (K + 1);
    const int nch = n_chunks(V);
    return align256(rows * nch * sizeof(ChunkStat)) + align256(rows * sizeof(RowInfo)) +
           align256((size_t)R * sizeof(DrawInfo)) + align256((size_t)R * nch * sizeof(double)) +
           align256(rows * nch * sizeof(double));
}

// exp2 on the transcendental unit (v_exp_f32)
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
// NaN-propagating maximum without operand canonicalisation (v_maximum3_f32)
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

template <bool BF16>
__device__ __forceinline__ float load_logit(const void* base, int64_t i) {
    if (BF16) return bf16_to_f32(((const uint16_t*)base)[i]);
    return ((const float*)base)[i];
}

// ---------------------------------------------------------------- wave chunks
//
// A wave reads a chunk as 16-byte words: lane l's word q covers entries
// v0 + (q * 64 + l) * G .. + G - 1 (G = 8 bf16 or 4 fp32 entries), so every
// load instruction of the wave reads one contiguous kilobyte.  Lane-local
// entry k = q * G + j; the entries of one lane increase with k.
template <bool BF16>
struct WaveChunk {
    static constexpr int G = BF16 ? 8 : 4;
    static constexpr int NW = kLanePer / G;  // words per lane
    u32x4 w[NW];
};

template <bool BF16>
__device__ __forceinline__ int wc_index(int v0, int lane, int k) {
    constexpr int G = WaveChunk<BF16>::G;
    return v0 + ((k / G) * kLanes + lane) * G + (k % G);
}

// 16-byte loads of the chunk at v0 of a row of V entries (V a whole number of
// words, the row 16-byte aligned).  Words at or past the row's end re-read its
// last word, so every load stays inside the row; wc_mask() then clears them.
template <bool BF16>
__device__ __forceinline__ void wc_load(const void* row, int v0, int V, int lane, WaveChunk<BF16>& c) {
    constexpr int G = WaveChunk<BF16>::G;
    constexpr int esz = BF16 ? 2 : 4;
    const int last = V - G;
#pragma unroll
    for (int q = 0; q < WaveChunk<BF16>::NW; ++q) {
        const int e0 = min(v0 + (q * kLanes + lane) * G, last);
        c.w[q] = __builtin_nontemporal_load((const u32x4*)((const char*)row + (size_t)e0 * esz));
    }
}

// entries at or past v1 (a row's last, partial chunk) become `fill`
template <bool BF16>
__device__ __forceinline__ void wc_mask(float* x, int v0, int v1, int lane, float fill) {
#pragma unroll
    for (int k = 0; k < kLanePer; ++k)
        if (wc_index<BF16>(v0, lane, k) >= v1) x[k] = fill;
}

template <bool BF16>
__device__ __forceinline__ void wc_unpack(const WaveChunk<BF16>& c, float* x) {
    if constexpr (BF16) {
#pragma unroll
        for (int q = 0; q < WaveChunk<BF16>::NW; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[q * 8 + 2 * e] = __uint_as_float(c.w[q][e] << 16);
                x[q * 8 + 2 * e + 1] = __uint_as_float(c.w[q][e] & 0xffff0000u);
            }
    } else {
#pragma unroll
        for (int q = 0; q < WaveChunk<BF16>::NW; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) x[q * 4 + e] = __uint_as_float(c.w[q][e]);
    }
}

// Entries of [v0, v1) in the same layout with per-entry loads of a clamped
// index (all in flight at once); entries at or past v1 get `fill`.  Used for a
// row's last, partial chunk and for rows that are not 16-byte aligned.
template <bool BF16>
__device__ __forceinline__ void wc_load_slow(const void* row, int v0, int v1, int lane, float fill,
                                             float* x) {
#pragma unroll
    for (int k = 0; k < kLanePer; ++k) {
        const int v = wc_index<BF16>(v0, lane, k);
        const float xv = load_logit<BF16>(row, min(v, v1 - 1));
        x[k] = v < v1 ? xv : fill;
    }
}

// Draft probabilities (fp32) at the entries of a logits chunk, clamped like
// wc_load().
template <bool BF16>
__device__ __forceinline__ void wc_load_draft(const float* pd, int v0, int V, int lane, f32x4* d) {
    constexpr int G = WaveChunk<BF16>::G;
    const int last = V - G;
#pragma unroll
    for (int q = 0; q < WaveChunk<BF16>::NW; ++q) {
        const int e0 = min(v0 + (q * kLanes + lane) * G, last);
#pragma unroll
        for (int h = 0; h < G / 4; ++h)
            d[q * (G / 4) + h] = __builtin_nontemporal_load((const f32x4*)(pd + e0 + 4 * h));
    }
}

template <bool BF16>
__device__ __forceinline__ void wc_load_draft_slow(const float* pd, int v0, int v1, int lane,
                                                   float* q) {
#pragma unroll
    for (int k = 0; k < kLanePer; ++k) {
        const int v = wc_index<BF16>(v0, lane, k);
        const float qv = pd[min(v, v1 - 1)];
        q[k] = v < v1 ? qv : 0.0f;
    }
}

// ---------------------------------------------------------------- rowpass

// Statistics of one chunk held in x[] (lane layout above), written by lane 0.
template <bool BF16, bool GREEDY>
__device__ __forceinline__ void chunk_stat(const float* x, int v0, int lane, float scale2,
                                           ChunkStat* out) {
    if (GREEDY) {
        // lane-local max; the strict comparison keeps the lowest entry on ties
        float best = x[0];
        int bk = 0;
#pragma unroll
        for (int k = 1; k < kLanePer; ++k)
            if (x[k] > best) { best = x[k]; bk = k; }
        int arg = wc_index<BF16>(v0, lane, bk);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const float ob = __shfl_xor(best, o, kLanes);
            const int oa = __shfl_xor(arg, o, kLanes);
            if (ob > best || (ob == best && oa < arg)) { best = ob; arg = oa; }
        }
        if (lane == 0) *out = ChunkStat{best, 0.0f, arg, 0};
    } else {
        // max of the raw logits (the scale is positive), then the sum of
        // exp2(scale2 * x - m) with m the scaled max
        float mx = x[0];
#pragma unroll
        for (int k = 1; k < kLanePer; ++k) mx = vmax(mx, x[k]);
        const float m = mx * scale2;
        float sum = 0.0f;
        if (m > -__builtin_huge_valf()) {
#pragma unroll
            for (int k = 0; k < kLanePer; ++k) sum += fexp2(__builtin_fmaf(x[k], scale2, -m));
        }
        const float wm = wave_max(m);
        sum = (m > -__builtin_huge_valf()) ? sum * fexp2(m - wm) : 0.0f;
        sum = wave_sum(sum);
        if (lane == 0) *out = ChunkStat{wm, sum, 0, 0};
    }
}

// Stochastic mode also marks every row it covers as owned by no request
// (RowInfo req = -1); resolve then claims the rows of the well-formed requests,
// so rows that no well-formed request owns read as such in the rate pass.
template <bool BF16, bool GREEDY, bool VEC>
__global__ __launch_bounds__(kBlk) void acc_rowpass(
    const void* __restrict__ logits, int64_t ld, const int32_t* __restrict__ cu_q, int R, int V,
    int max_rows, float scale2, ChunkStat* __restrict__ stats, RowInfo* __restrict__ rows) {
    const int nch = n_chunks(V);
    const int items = clamp_rows(cu_q[R], max_rows) * nch;
    const int lane = threadIdx.x & (kLanes - 1);
    const size_t row_bytes = (size_t)ld * (BF16 ? 2 : 4);
    auto row_of = [&](int i) {
        return (const void*)((const char*)logits + (size_t)(i / nch) * row_bytes);
    };
    auto load = [&](int i, WaveChunk<BF16>& c) {
        if (VEC) wc_load<BF16>(row_of(i), (i % nch) * kChunk, V, lane, c);
    };
    // each wave walks a contiguous range of (row, chunk) items, i.e. whole
    // stretches of logit rows.  One register buffer: a chunk's words are
    // unpacked into x as soon as they land, and the buffer is refilled with
    // the next chunk right away, so its loads are in flight while this chunk
    // is reduced (fewer registers than two buffers, so more waves per SIMD)
    const int nwv = gridDim.x * kWaves;
    const int per = (items + nwv - 1) / nwv;
    int it = (blockIdx.x * kWaves + wave_id()) * per;
    const int end = min(items, it + per);
    WaveChunk<BF16> A;
    if (it < end) load(it, A);
    for (; it < end; ++it) {
        const int v0 = (it % nch) * kChunk;
        const int v1 = min(V, v0 + kChunk);
        float x[kLanePer];
        if (VEC) {
            wc_unpack<BF16>(A, x);
            if (it + 1 < end) load(it + 1, A);
            if (v1 < v0 + kChunk) wc_mask<BF16>(x, v0, v1, lane, -__builtin_huge_valf());
        } else {
            wc_load_slow<BF16>(row_of(it), v0, v1, lane, -__builtin_huge_valf(), x);
        }
        chunk_stat<BF16, GREEDY>(x, v0, lane, scale2, stats + it);
        if (!GREEDY && lane == 0 && v0 == 0) rows[it / nch] = RowInfo{0.0f, 0.0f, -1, -1};
    }
}

// ---------------------------------------------------------------- resolve

// Row statistics from the chunk statistics: one wave per row, lanes over
// chunks.  A lane folds its chunks in order (stat_absorb), then the wave
// combines the lanes (stat_combine).
template <bool GREEDY>
__device__ __forceinline__ void stat_absorb(const ChunkStat& x, float& a, float& b, int& i) {
    if (GREEDY) {
        if (x.a > a || (x.a == a && x.arg < i)) { a = x.a; i = x.arg; }
    } else if (x.a > -__builtin_huge_valf()) {
        if (x.a > a) { b = b * exp2f(a - x.a) + x.b; a = x.a; }
        else b += x.b * exp2f(x.a - a);
    }
}

template <bool GREEDY>
__device__ __forceinline__ void stat_combine(float& a, float& b, int& i) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float oa = __shfl_xor(a, o, kLanes);
        const float ob = __shfl_xor(b, o, kLanes);
        const int oi = __shfl_xor(i, o, kLanes);
        if (GREEDY) {
            if (oa > a || (oa == a && oi < i)) { a = oa; i = oi; }
        } else {
            const float m = fmaxf(a, oa);
            float nb = 0.0f;
            if (a > -__builtin_huge_valf()) nb += b * exp2f(a - m);
            if (oa > -__builtin_huge_valf()) nb += ob * exp2f(oa - m);
            a = m;
            b = nb;
        }
    }
}

template <bool GREEDY>
__device__ __forceinline__ void row_stats(const ChunkStat* st, int nch, float& A, float& B,
                                          int& arg) {
    const int lane = threadIdx.x & (kLanes - 1);
    float a = -__builtin_huge_valf(), b = 0.0f;
    int i = 0x7fffffff;
    for (int c = lane; c < nch; c += kLanes) stat_absorb<GREEDY>(st[c], a, b, i);
    stat_combine<GREEDY>(a, b, i);
    A = a;
    B = b;
    arg = i;
}

constexpr int kResolveRows = (65 + kWaves - 1) / kWaves;  // rows per wave (K <= 64)

template <bool BF16, bool GREEDY>
__global__ __launch_bounds__(kBlk) void acc_resolve(
    const int32_t* __restrict__ draft_tok, const float* __restrict__ draft_p,
    const void* __restrict__ logits, int64_t ld, const float* __restrict__ u,
    const int32_t* __restrict__ cu_q, int R, int K, int V, float scale2,
    const ChunkStat* __restrict__ stats, RowInfo* __restrict__ rows, DrawInfo* __restrict__ draw,
    int32_t* __restrict__ accepted_len, int32_t* __restrict__ next_tok) {
    __shared__ int s_rej[65];
    __shared__ int s_arg[65];
    __shared__ int s_tok[64];
    __shared__ float s_M[65], s_S[65];
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kLanes - 1);
    const int wave = tid / kLanes;
    const int nch = n_chunks(V);
    // the drafts are loaded together with the request's row range
    if (tid < K) s_tok[tid] = draft_tok[(int64_t)r * K + tid];
    const int row0 = cu_q[r];
    const int l = cu_q[r + 1] - row0 - 1;
    __syncthreads();
    // the request's rows must lie inside the rows the row pass covered (and the
    // caller sized): [0, min(cu_q[R], R * (K + 1)))
    if (l < 0 || l > K || row0 < 0 ||
        (int64_t)row0 + l + 1 > (int64_t)clamp_rows(cu_q[R], R * (K + 1))) {
        if (tid == 0) {
            accepted_len[r] = -1;
            next_tok[r] = -1;
            if (!GREEDY) draw[r] = DrawInfo{0, 0, 0, 0, 0.0f, 0.0f, {0, 0}};
        }
        return;
    }
    const size_t esz = BF16 ? 2 : 4;
    // row t's results: statistics and accept test, kept by lane `ln`
    auto finish = [&](int t, int ln, float A, float B, int arg, bool test, float y, float pd,
                      float uu) {
        if (lane != ln) return;
        int rej = 0;
        if (GREEDY) {
            if (t < l) rej = s_tok[t] != arg;
            s_arg[t] = arg;
        } else {
            rows[row0 + t] = RowInfo{A, B, r, t};
            s_M[t] = A;
            s_S[t] = B;
            if (t < l) {
                if (!test) {
                    rej = 1;  // draft token outside the vocabulary
                } else {
                    const float pt = exp2f(y - A) / B;
                    const float ratio = pd > 0.0f ? pt / pd : __builtin_huge_valf();
                    rej = !(uu < ratio);
                }
            }
        }
        s_rej[t] = rej;
    };
    // the tested draft's target logit, draft probability and uniform of row t
    auto gather = [&](int t, bool& test, float& y, float& pd, float& uu) {
        const int x = t < l ? s_tok[t] : -1;
        test = !GREEDY && t < l && x >= 0 && x < V;
        y = pd = uu = 0.0f;
        if (test) {
            const void* rp = (const char*)logits + (size_t)(row0 + t) * (size_t)ld * esz;
            y = load_logit<BF16>(rp, x) * scale2;
            pd = draft_p[((int64_t)r * K + t) * V + x];
            uu = u[(int64_t)r * (K + 1) + t];
        }
    };
    if (nch <= kLanes) {
        // one chunk per lane: the chunk statistics of every row of this wave
        // (t = wave + 4 j) and, on lane j, row t's test inputs are all in
        // flight at once
        ChunkStat xs[kResolveRows];
#pragma unroll
        for (int j = 0; j < kResolveRows; ++j) {
            const int t = wave + kWaves * j;
            if (t <= l && lane < nch) xs[j] = stats[(int64_t)(row0 + t) * nch + lane];
        }
        const int tj = wave + kWaves * lane;
        bool test = false;
        float y = 0.0f, pd = 0.0f, uu = 0.0f;
        if (lane < kResolveRows && tj <= l) gather(tj, test, y, pd, uu);
#pragma unroll
        for (int j = 0; j < kResolveRows; ++j) {
            const int t = wave + kWaves * j;
            if (t > l) break;
            float a = -__builtin_huge_valf(), b = 0.0f;
            int i = 0x7fffffff;
            if (lane < nch) stat_absorb<GREEDY>(xs[j], a, b, i);
            stat_combine<GREEDY>(a, b, i);
            finish(t, j, a, b, i, test, y, pd, uu);
        }
    } else {
        for (int t = wave; t <= l; t += kWaves) {
            bool test = false;
            float y = 0.0f, pd = 0.0f, uu = 0.0f;
            if (lane == 0) gather(t, test, y, pd, uu);
            float A, B;
            int arg;
            row_stats<GREEDY>(stats + (int64_t)(row0 + t) * nch, nch, A, B, arg);
            finish(t, 0, A, B, arg, test, y, pd, uu);
        }
    }
    __syncthreads();
    if (tid == 0) {
        int acc = l;
        for (int t = 0; t < l; ++t)
            if (s_rej[t]) { acc = t; break; }
        accepted_len[r] = acc;
        if (GREEDY) next_tok[r] = s_arg[acc];
        else draw[r] = DrawInfo{acc < l ? 2 : 1, row0 + acc, acc, 0, s_M[acc], s_S[acc], {0, 0}};
    }
}

// ---------------------------------------------------------------- residual masses

// One wave per (request, chunk): the mass of max(0, p_t - p_d) of the
// rejected row, for requests that rejected (the others return at once).
template <bool BF16, bool VEC>
__global__ __launch_bounds__(kBlk) void acc_resid(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld, int R, int K,
    int V, float scale2, const DrawInfo* __restrict__ draw, double* __restrict__ mass) {
    const int nch = n_chunks(V);
    const int lane = threadIdx.x & (kLanes - 1);
    const int it = blockIdx.x * kWaves + wave_id();
    if (it >= R * nch) return;
    const int r = it / nch;
    const int c = it - r * nch;
    const DrawInfo d = draw[r];
    if (d.kind != 2) return;
    const int v0 = c * kChunk;
    const int v1 = min(V, v0 + kChunk);
    const void* rp = (const char*)logits + (size_t)d.row * (size_t)ld * (BF16 ? 2 : 4);
    const float* pd = draft_p + ((int64_t)r * K + d.t) * V;
    const float invS = 1.0f / d.S;
    float acc = 0.0f;
    if (VEC) {
        WaveChunk<BF16> xc;
        f32x4 qd[kLanePer / 4];
        wc_load<BF16>(rp, v0, V, lane, xc);
        wc_load_draft<BF16>(pd, v0, V, lane, qd);
        float x[kLanePer];
        wc_unpack<BF16>(xc, x);
        // entries past v1: x = -inf gives p_t = 0 and the term max(0, -p_d) = 0
        if (v1 < v0 + kChunk) wc_mask<BF16>(x, v0, v1, lane, -__builtin_huge_valf());
#pragma unroll
        for (int k = 0; k < kLanePer; ++k) {
            const float pt = fexp2(__builtin_fmaf(x[k], scale2, -d.M)) * invS;
            acc += fmaxf(pt - qd[k / 4][k % 4], 0.0f);
        }
    } else {
        float x[kLanePer], q[kLanePer];
        wc_load_slow<BF16>(rp, v0, v1, lane, -__builtin_huge_valf(), x);
        wc_load_draft_slow<BF16>(pd, v0, v1, lane, q);
#pragma unroll
        for (int k = 0; k < kLanePer; ++k) {
            // entries past v1 have x = -inf: exp2 gives 0 and the term vanishes
            const float pt = fexp2(__builtin_fmaf(x[k], scale2, -d.M)) * invS;
            acc += fmaxf(pt - q[k], 0.0f);
        }
    }
    const double w = wave_sum_f64((double)acc);
    if (lane == 0) mass[it] = w;
}

// ---------------------------------------------------------------- draw

template <bool BF16>
__global__ __launch_bounds__(kBlk) void acc_draw(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld,
    const float* __restrict__ u, int R, int K, int V, float scale2,
    const ChunkStat* __restrict__ stats, const DrawInfo* __restrict__ draw,
    const double* __restrict__ mass, int32_t* __restrict__ next_tok) {
    __shared__ double s_w[kMaxChunks];
    __shared__ int s_chunk;
    __shared__ double s_thr;
    __shared__ int s_kind;
    __shared__ double s_scan[kWaves];
    __shared__ int s_pick;
    __shared__ int s_last;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kLanes - 1);
    const int wave = tid / kLanes;
    const int nch = n_chunks(V);
    // the residual chunk masses (nch <= kBlk) and u are loaded together with
    // the draw record
    const double mw = tid < nch ? mass[(int64_t)r * nch + tid] : 0.0;
    const double uu = (double)u[(int64_t)r * (K + 1) + K];
    const DrawInfo d = draw[r];
    if (d.kind == 0) return;
    const ChunkStat* st = stats + (int64_t)d.row * nch;
    // chunk masses, in the units of the entry masses used below
    int kind = d.kind;
    if (kind == 2) {
        double t = wave_sum_f64(mw);
        if (lane == 0) s_scan[wave] = t;
        __syncthreads();
        double tot = 0.0;
        for (int q = 0; q < kWaves; ++q) tot += s_scan[q];
        if (!(tot > 0.0)) kind = 1;  // empty residual: draw from the target row
        __syncthreads();
    }
    if (tid < nch) {
        if (kind == 2) {
            s_w[tid] = mw;
        } else {
            const ChunkStat x = st[tid];
            s_w[tid] = x.a > -__builtin_huge_valf() ? (double)x.b * (double)exp2f(x.a - d.M) : 0.0;
        }
    }
    __syncthreads();
    if (wave == 0) {
        // the chunk where the running mass first exceeds u * total: lane l
        // holds chunks 4l .. 4l + 3 (nch <= 256)
        double w4[4], loc = 0.0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int c = 4 * lane + k;
            w4[k] = c < nch ? s_w[c] : 0.0;
            loc += w4[k];
        }
        double incl = loc;
#pragma unroll
        for (int o = 1; o < kLanes; o <<= 1) {
            const double t = __shfl_up(incl, o, kLanes);
            if (lane >= o) incl += t;
        }
        const double tot = __shfl(incl, kLanes - 1, kLanes);
        const double thr = uu * tot;
        int lastpos = -1;  // last non-empty chunk of this lane
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (w4[k] > 0.0) lastpos = 4 * lane + k;
        // (a lane with no mass never holds the crossing, whatever the rounding)
        const unsigned long long hit = __ballot(incl > thr && loc > 0.0);
        if (hit) {
            // the first lane whose running mass passes thr holds the chunk
            if (lane == (int)__builtin_ctzll(hit)) {
                double cum = incl - loc;
                int pick = -1;
                double before = 0.0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    if (pick < 0 && cum + w4[k] > thr) { pick = 4 * lane + k; before = cum; }
                    cum += w4[k];
                }
                if (pick < 0) {  // summation order: the lane's last non-empty chunk
                    pick = lastpos;
                    before = cum - w4[pick - 4 * lane];
                }
                s_chunk = pick;
                s_thr = thr - before;
            }
        } else {
            // rounding pushed u * total past the end: the last non-empty chunk
            const int lp = __reduce_max_sync(~0ull, lastpos);
            if (lane == 0) {
                const int pick = lp >= 0 ? lp : 0;
                s_chunk = pick;
                s_thr = thr - (tot - s_w[pick]);
            }
        }
        if (lane == 0) {
            s_kind = kind;
            s_pick = 0x7fffffff;
            s_last = -1;
        }
    }
    __syncthreads();
    const int c = s_chunk;
    kind = s_kind;
    const double thr = s_thr;
    const int v0 = c * kChunk;
    const int v1 = min(V, v0 + kChunk);
    const size_t esz = BF16 ? 2 : 4;
    const void* rp = (const char*)logits + (size_t)d.row * (size_t)ld * esz;
    const float* pd = draft_p + ((int64_t)r * K + d.t) * V;
    const float invS = 1.0f / d.S;
    // this thread's contiguous slice [first, first + kThreadPer) of the chunk
    const int first = v0 + tid * kThreadPer;
    float x[kThreadPer], q[kThreadPer];
    const bool full = first + kThreadPer <= v1;
    const bool xvec = full && ((uintptr_t)((const char*)rp + (size_t)first * esz) % 16 == 0);
    if (xvec && BF16) {
        const u32x4* p4 = (const u32x4*)((const uint16_t*)rp + first);
#pragma unroll
        for (int k = 0; k < kThreadPer / 8; ++k) {
            const u32x4 w = p4[k];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[8 * k + 2 * e] = __uint_as_float(w[e] << 16);
                x[8 * k + 2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
            }
        }
    } else if (xvec) {
        const f32x4* p4 = (const f32x4*)((const float*)rp + first);
#pragma unroll
        for (int k = 0; k < kThreadPer / 4; ++k) {
            const f32x4 w = p4[k];
            x[4 * k] = w[0]; x[4 * k + 1] = w[1]; x[4 * k + 2] = w[2]; x[4 * k + 3] = w[3];
        }
    } else {
#pragma unroll
        for (int e = 0; e < kThreadPer; ++e) {
            const float xv = load_logit<BF16>(rp, min(first + e, v1 - 1));
            x[e] = first + e < v1 ? xv : -__builtin_huge_valf();
        }
    }
    if (kind == 2) {
        if (full && ((uintptr_t)(pd + first) % 16 == 0)) {
            const f32x4* p4 = (const f32x4*)(pd + first);
#pragma unroll
            for (int k = 0; k < kThreadPer / 4; ++k) {
                const f32x4 w = p4[k];
                q[4 * k] = w[0]; q[4 * k + 1] = w[1]; q[4 * k + 2] = w[2]; q[4 * k + 3] = w[3];
            }
        } else {
#pragma unroll
            for (int e = 0; e < kThreadPer; ++e) {
                const float qv = pd[min(first + e, v1 - 1)];
                q[e] = first + e < v1 ? qv : 0.0f;
            }
        }
    }
    float wv[kThreadPer];
    double loc = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int e = 0; e < kThreadPer; ++e) {
        float m;
        if (kind == 2) m = fmaxf(fexp2(__builtin_fmaf(x[e], scale2, -d.M)) * invS - q[e], 0.0f);
        else m = fexp2(__builtin_fmaf(x[e], scale2, -d.M));
        if (first + e >= v1) m = 0.0f;
        wv[e] = m;
        loc += (double)m;
        if (m > 0.0f) lastpos = first + e;
    }
    // exclusive scan of the per-thread sums over the block
    double incl = loc;
#pragma unroll
    for (int o = 1; o < kLanes; o <<= 1) {
        const double t = __shfl_up(incl, o, kLanes);
        if (lane >= o) incl += t;
    }
    if (lane == kLanes - 1) s_scan[wave] = incl;
    __syncthreads();
    double pre = incl - loc;
    for (int k = 0; k < wave; ++k) pre += s_scan[k];
    // the smallest index whose running mass exceeds thr; threads past the
    // crossing also propose a candidate, and the minimum wins
    if (pre + loc > thr) {
        double cum = pre;
        for (int e = 0; e < kThreadPer; ++e) {
            cum += (double)wv[e];
            if (cum > thr) { atomicMin(&s_pick, first + e); break; }
        }
    }
    if (lastpos >= 0) atomicMax(&s_last, lastpos);
    __syncthreads();
    if (tid == 0) {
        int v = s_pick;
        if (v == 0x7fffffff) v = s_last >= 0 ? s_last : v0;
        next_tok[r] = v;
    }
}

// ---------------------------------------------------------------- analytic rate

// One wave per (row, chunk): sum_v min(p_t, p_d) over the chunk for rows that
// test a draft; other rows return at once.
template <bool BF16, bool VEC>
__global__ __launch_bounds__(kBlk) void acc_rate_pass(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld,
    const int32_t* __restrict__ cu_q, int R, int K, int V, float scale2,
    const RowInfo* __restrict__ rows, double* __restrict__ part) {
    const int nch = n_chunks(V);
    const int lane = threadIdx.x & (kLanes - 1);
    const int it = blockIdx.x * kWaves + wave_id();
    if (it >= clamp_rows(cu_q[R], R * (K + 1)) * nch) return;
    const int row = it / nch;
    const int c = it - row * nch;
    const RowInfo ri = rows[row];
    const int r = ri.req;
    // rows of malformed requests and bonus rows carry no draft
    if (r < 0 || r >= R || ri.t < 0 || ri.t >= K) return;
    const int ql = cu_q[r + 1] - cu_q[r];
    if (ri.t >= ql - 1) return;
    const int v0 = c * kChunk;
    const int v1 = min(V, v0 + kChunk);
    const void* rp = (const char*)logits + (size_t)row * (size_t)ld * (BF16 ? 2 : 4);
    const float* pd = draft_p + ((int64_t)r * K + ri.t) * V;
    const float invS = 1.0f / ri.S;
    float acc = 0.0f;
    if (VEC) {
        WaveChunk<BF16> xc;
        f32x4 qd[kLanePer / 4];
        wc_load<BF16>(rp, v0, V, lane, xc);
        wc_load_draft<BF16>(pd, v0, V, lane, qd);
        float x[kLanePer];
        wc_unpack<BF16>(xc, x);
        // entries past v1: x = -inf gives min(0, p_d) = 0
        if (v1 < v0 + kChunk) wc_mask<BF16>(x, v0, v1, lane, -__builtin_huge_valf());
#pragma unroll
        for (int k = 0; k < kLanePer; ++k)
            acc += fminf(fexp2(__builtin_fmaf(x[k], scale2, -ri.M)) * invS, qd[k / 4][k % 4]);
    } else {
        float x[kLanePer], q[kLanePer];
        wc_load_slow<BF16>(rp, v0, v1, lane, -__builtin_huge_valf(), x);
        wc_load_draft_slow<BF16>(pd, v0, v1, lane, q);
#pragma unroll
        for (int k = 0; k < kLanePer; ++k)
            acc += fminf(fexp2(__builtin_fmaf(x[k], scale2, -ri.M)) * invS, q[k]);
    }
    const double w = wave_sum_f64((double)acc);
    if (lane == 0) part[it] = w;
}

__global__ __launch_bounds__(kBlk) void acc_rate_final(
    const int32_t* __restrict__ cu_q, int R, int V, int max_rows, const RowInfo* __restrict__ rows,
    const double* __restrict__ part, float* __restrict__ rate) {
    const int nch = n_chunks(V);
    const int total = clamp_rows(cu_q[R], max_rows);
    for (int row = blockIdx.x * blockDim.x + threadIdx.x; row < total;
         row += gridDim.x * blockDim.x) {
        const RowInfo ri = rows[row];
        if (ri.req < 0 || ri.req >= R || ri.t < 0) { rate[row] = -1.0f; continue; }
        const int ql = cu_q[ri.req + 1] - cu_q[ri.req];
        if (ri.t >= ql - 1) { rate[row] = -1.0f; continue; }
        double t = 0.0;
        for (int c = 0; c < nch; ++c) t += part[(int64_t)row * nch + c];
        rate[row] = (float)t;
    }
}

// ---------------------------------------------------------------- launch

// resident workgroups of a kernel on the whole device (persistent grids)
static int resident_blocks(const void* fn, int cus) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlk, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    return per_cu * cus;
}

template <bool BF16>
static hipError_t launch_typed(const AcceptArgs& a, void* ws, hipStream_t s) {
    const AccWs w = carve(ws, a.R, a.K, a.V);
    const int nch = n_chunks(a.V);
    const float scale2 = a.inv_temp * kLog2e;
    const bool greedy = a.draft_p == nullptr && a.u == nullptr;
    const size_t esz = BF16 ? 2 : 4;
    // 16-byte words: aligned rows made of whole words (else per-entry loads)
    const int G = BF16 ? 8 : 4;
    const bool vec = ((uintptr_t)a.logits % 16 == 0) && ((size_t)a.ld * esz) % 16 == 0 &&
                     a.V % G == 0;
    const int max_rows = a.R * (a.K + 1);
    const int64_t wave_items = (int64_t)max_rows * nch;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const dim3 blk(kBlk);
    // the row pass runs as many persistent workgroups as are resident at once
    const void* rowpass = greedy ? (vec ? (const void*)acc_rowpass<BF16, true, true>
                                        : (const void*)acc_rowpass<BF16, true, false>)
                                 : (vec ? (const void*)acc_rowpass<BF16, false, true>
                                        : (const void*)acc_rowpass<BF16, false, false>);
    const int pgrid = (int)std::max<int64_t>(
        1, std::min<int64_t>((wave_items + kWaves - 1) / kWaves, resident_blocks(rowpass, cus)));
#define DS_ROWPASS(G, VV)                                                                    \
    hipLaunchKernelGGL((acc_rowpass<BF16, G, VV>), dim3(pgrid), blk, 0, s, a.logits, a.ld, \
                       a.cu_q, a.R, a.V, max_rows, scale2, w.stats, w.rows)
    if (greedy) { if (vec) DS_ROWPASS(true, true); else DS_ROWPASS(true, false); }
    else { if (vec) DS_ROWPASS(false, true); else DS_ROWPASS(false, false); }
#undef DS_ROWPASS
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (greedy) {
        hipLaunchKernelGGL((acc_resolve<BF16, true>), dim3(a.R), blk, 0, s, a.draft_tok,
                           a.draft_p, a.logits, a.ld, a.u, a.cu_q, a.R, a.K, a.V, scale2,
                           w.stats, w.rows, w.draw, a.accepted_len, a.next_tok);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((acc_resolve<BF16, false>), dim3(a.R), blk, 0, s, a.draft_tok, a.draft_p,
                       a.logits, a.ld, a.u, a.cu_q, a.R, a.K, a.V, scale2, w.stats, w.rows,
                       w.draw, a.accepted_len, a.next_tok);
    // draft rows start at multiples of V floats: 16-byte aligned when V % 4 == 0
    // (implied by whole logit words)
    const bool pdvec = vec && ((uintptr_t)a.draft_p % 16) == 0;
    const int rgrid = (int)(((int64_t)a.R * nch + kWaves - 1) / kWaves);
    if (pdvec)
        hipLaunchKernelGGL((acc_resid<BF16, true>), dim3(rgrid), blk, 0, s, a.draft_p, a.logits,
                           a.ld, a.R, a.K, a.V, scale2, w.draw, w.mass);
    else
        hipLaunchKernelGGL((acc_resid<BF16, false>), dim3(rgrid), blk, 0, s, a.draft_p, a.logits,
                           a.ld, a.R, a.K, a.V, scale2, w.draw, w.mass);
    hipLaunchKernelGGL((acc_draw<BF16>), dim3(a.R), blk, 0, s, a.draft_p, a.logits, a.ld, a.u,
                       a.R, a.K, a.V, scale2, w.stats, w.draw, w.mass, a.next_tok);
    if (a.accept_rate) {
        const int qgrid = (int)std::max<int64_t>(1, (wave_items + kWaves - 1) / kWaves);
        if (pdvec)
            hipLaunchKernelGGL((acc_rate_pass<BF16, true>), dim3(qgrid), blk, 0, s, a.draft_p,
                               a.logits, a.ld, a.cu_q, a.R, a.K, a.V, scale2, w.rows, w.rate);
        else
            hipLaunchKernelGGL((acc_rate_pass<BF16, false>), dim3(qgrid), blk, 0, s, a.draft_p,
                               a.logits, a.ld, a.cu_q, a.R, a.K, a.V, scale2, w.rows, w.rate);
        const int fgrid = (int)std::max<int64_t>(
            1, std::min<int64_t>(((int64_t)max_rows + kBlk - 1) / kBlk, 1024));
        hipLaunchKernelGGL(acc_rate_final, dim3(fgrid), blk, 0, s, a.cu_q, a.R, a.V, max_rows,
                           w.rows, w.rate, a.accept_rate);
    }
    return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, void* ws, hipStream_t s) {
    return a.logit_bf16 ? launch_typed<true>(a, ws, s) : launch_typed<false>(a, ws, s);
}

}  // namespace dspark
