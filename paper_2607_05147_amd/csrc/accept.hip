// Speculative acceptance over the vocabulary on gfx950 (the left-to-right
// acceptance rule of the speculative-decoding background section).
//
// Kernels, in stream order:
//   rowpass  one pass over every verified logit row, in 8192-token chunks:
//            per chunk the max and argmax of the raw logits (greedy) or the max
//            and sum of exp2 of the scaled logits (stochastic).  HBM streaming;
//            a persistent grid walks (row, chunk) items.
//   resolve  one workgroup per request: per-row statistics from the chunk
//            statistics, the accept test of every draft (greedy match or
//            u < p_t(x) / p_d(x)), the first rejection, and what to draw from.
//   resid    stochastic requests with a rejection: per chunk, the mass of the
//            residual max(0, p_t - p_d) of the rejected row.
//   draw     one workgroup per stochastic request: inverse CDF at u[r, K] over
//            the chunk masses, then inside the selected chunk only.
//   rate     (optional) sum_v min(p_t, p_d) per tested row.
// Probabilities are evaluated in fp32 (exp2 of log2e-scaled logits); masses
// are accumulated in fp64 across threads and chunks.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace dspark {

constexpr int kAccThreads = 256;
constexpr int kChunk = 8192;                        // vocabulary entries per chunk
constexpr int kPerThread = kChunk / kAccThreads;    // 32
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxChunks = 128;                     // V <= 2^20

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct ChunkStat {
    float a;   // greedy: max raw logit      stochastic: max of scaled logit (log2 units)
    float b;   // greedy: unused             stochastic: sum exp2(y - a)
    int arg;   // greedy: argmax (lowest index on ties)
    int pad;
};

struct RowInfo {     // per verified row, written by resolve
    float M, S;      // row max (log2 units) and sum of exp2(y - M)
    int req, t;      // owning request and verify slot
};

struct DrawInfo {    // per request
    int kind;        // 0 none, 1 target row, 2 residual of a rejected row
    int row;         // flattened logit row
    int t;           // verify slot of that row
    int pad;
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

// ---------------------------------------------------------------- loading

template <bool BF16>
__device__ __forceinline__ float load_logit(const void* base, int64_t i) {
    if (BF16) return bf16_to_f32(((const uint16_t*)base)[i]);
    return ((const float*)base)[i];
}

// Element e of this thread within a chunk starting at v0, in the
// lane-interleaved layout used by the reductions: every 16-byte group of
// consecutive elements belongs to one thread and consecutive threads read
// consecutive groups, so each load instruction covers one contiguous span.
template <bool BF16>
__device__ __forceinline__ int ilv_index(int v0, int e) {
    constexpr int G = BF16 ? 8 : 4;  // elements per 16 bytes
    return v0 + (e / G) * (kAccThreads * G) + threadIdx.x * G + (e % G);
}

// Loads this thread's kPerThread logits of [v0, v1) (interleaved layout) into
// x[]; positions past v1 get -inf.  VEC: 16-byte loads for full chunks.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load_chunk(const void* row, int v0, int v1, float* x) {
    constexpr int G = BF16 ? 8 : 4;
    if (VEC && v0 + kChunk <= v1) {
        if (BF16) {
            const u32x4* p = (const u32x4*)((const uint16_t*)row + v0) + threadIdx.x;
#pragma unroll
            for (int q = 0; q < kPerThread / G; ++q) {
                const u32x4 w = __builtin_nontemporal_load(p + q * kAccThreads);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[q * 8 + 2 * e] = __uint_as_float(w[e] << 16);
                    x[q * 8 + 2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
                }
            }
        } else {
            const f32x4* p = (const f32x4*)((const float*)row + v0) + threadIdx.x;
#pragma unroll
            for (int q = 0; q < kPerThread / G; ++q) {
                const f32x4 w = __builtin_nontemporal_load(p + q * kAccThreads);
                x[q * 4 + 0] = w[0]; x[q * 4 + 1] = w[1]; x[q * 4 + 2] = w[2]; x[q * 4 + 3] = w[3];
            }
        }
    } else {
        // partial chunk: unconditional loads of a clamped index (all in flight at
        // once), then mask; a conditional load per element would serialize
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const int v = ilv_index<BF16>(v0, e);
            const float xv = load_logit<BF16>(row, min(v, v1 - 1));
            x[e] = v < v1 ? xv : -__builtin_huge_valf();
        }
    }
}

// Draft probabilities of the same interleaved positions.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load_draft(const float* pd, int v0, int v1, float* x) {
    if (VEC && v0 + kChunk <= v1) {
        constexpr int G = BF16 ? 8 : 4;
        const f32x4* p = (const f32x4*)(pd + v0);
#pragma unroll
        for (int q = 0; q < kPerThread / G; ++q) {
#pragma unroll
            for (int h = 0; h < G / 4; ++h) {
                // elements q*G*256 + tid*G + 4h .. +4
                const f32x4 w = __builtin_nontemporal_load(
                    p + (q * kAccThreads * G + threadIdx.x * G) / 4 + h);
                x[q * G + 4 * h + 0] = w[0]; x[q * G + 4 * h + 1] = w[1];
                x[q * G + 4 * h + 2] = w[2]; x[q * G + 4 * h + 3] = w[3];
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const int v = ilv_index<BF16>(v0, e);
            const float qv = pd[min(v, v1 - 1)];
            x[e] = v < v1 ? qv : 0.0f;
        }
    }
}

// ---------------------------------------------------------------- rowpass

template <bool BF16, bool GREEDY, bool VEC>
__global__ __launch_bounds__(kAccThreads) void acc_rowpass(
    const void* __restrict__ logits, int64_t ld, const int32_t* __restrict__ cu_q, int R, int V,
    int max_rows, float scale2, ChunkStat* __restrict__ stats) {
    __shared__ float s_a[kAccThreads / DSPARK_WAVE];
    __shared__ float s_b[kAccThreads / DSPARK_WAVE];
    __shared__ int s_i[kAccThreads / DSPARK_WAVE];
    const int nch = n_chunks(V);
    const int64_t items = (int64_t)clamp_rows(cu_q[R], max_rows) * nch;
    const int lane = threadIdx.x & (DSPARK_WAVE - 1);
    const int wave = threadIdx.x / DSPARK_WAVE;
    const size_t esz = BF16 ? 2 : 4;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int64_t row = it / nch;
        const int c = (int)(it - row * nch);
        const int v0 = c * kChunk;
        const int v1 = min(V, v0 + kChunk);
        const void* rp = (const char*)logits + (size_t)row * (size_t)ld * esz;
        float x[kPerThread];
        load_chunk<BF16, VEC>(rp, v0, v1, x);
        if (GREEDY) {
            // thread-local max/argmax, lowest index among equal values
            float best = -__builtin_huge_valf();
            int arg = 0x7fffffff;
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) {
                const int v = ilv_index<BF16>(v0, e);
                if (v < v1 && (x[e] > best || (x[e] == best && v < arg))) { best = x[e]; arg = v; }
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                const float ob = __shfl_xor(best, o, DSPARK_WAVE);
                const int oa = __shfl_xor(arg, o, DSPARK_WAVE);
                if (ob > best || (ob == best && oa < arg)) { best = ob; arg = oa; }
            }
            if (lane == 0) { s_a[wave] = best; s_i[wave] = arg; }
            __syncthreads();
            if (threadIdx.x == 0) {
                float b = s_a[0];
                int a = s_i[0];
                for (int w = 1; w < kAccThreads / DSPARK_WAVE; ++w)
                    if (s_a[w] > b || (s_a[w] == b && s_i[w] < a)) { b = s_a[w]; a = s_i[w]; }
                stats[row * nch + c] = ChunkStat{b, 0.0f, a, 0};
            }
            __syncthreads();
        } else {
            float m = -__builtin_huge_valf();
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) { x[e] *= scale2; m = fmaxf(m, x[e]); }
            float s = 0.0f;
            if (m > -__builtin_huge_valf()) {
#pragma unroll
                for (int e = 0; e < kPerThread; ++e) s += exp2f(x[e] - m);
            }
            const float wm = wave_max(m);
            s = (m > -__builtin_huge_valf()) ? s * exp2f(m - wm) : 0.0f;
            s = wave_sum(s);
            if (lane == 0) { s_a[wave] = wm; s_b[wave] = s; }
            __syncthreads();
            if (threadIdx.x == 0) {
                float M = s_a[0];
                for (int w = 1; w < kAccThreads / DSPARK_WAVE; ++w) M = fmaxf(M, s_a[w]);
                float S = 0.0f;
                for (int w = 0; w < kAccThreads / DSPARK_WAVE; ++w)
                    if (s_a[w] > -__builtin_huge_valf()) S += s_b[w] * exp2f(s_a[w] - M);
                stats[row * nch + c] = ChunkStat{M, S, 0, 0};
            }
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------- resolve

// Row statistics from the chunk statistics: one wave per row, lanes over chunks.
template <bool GREEDY>
__device__ __forceinline__ void row_stats(const ChunkStat* st, int nch, float& A, float& B,
                                          int& arg) {
    const int lane = threadIdx.x & (DSPARK_WAVE - 1);
    float a = -__builtin_huge_valf(), b = 0.0f;
    int i = 0x7fffffff;
    for (int c = lane; c < nch; c += DSPARK_WAVE) {
        const ChunkStat x = st[c];
        if (GREEDY) {
            if (x.a > a || (x.a == a && x.arg < i)) { a = x.a; i = x.arg; }
        } else if (x.a > -__builtin_huge_valf()) {
            if (x.a > a) { b = b * exp2f(a - x.a) + x.b; a = x.a; }
            else b += x.b * exp2f(x.a - a);
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float oa = __shfl_xor(a, o, DSPARK_WAVE);
        const float ob = __shfl_xor(b, o, DSPARK_WAVE);
        const int oi = __shfl_xor(i, o, DSPARK_WAVE);
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
    A = a;
    B = b;
    arg = i;
}

template <bool BF16, bool GREEDY>
__global__ __launch_bounds__(kAccThreads) void acc_resolve(
    const int32_t* __restrict__ draft_tok, const float* __restrict__ draft_p,
    const void* __restrict__ logits, int64_t ld, const float* __restrict__ u,
    const int32_t* __restrict__ cu_q, int R, int K, int V, float scale2,
    const ChunkStat* __restrict__ stats, RowInfo* __restrict__ rows, DrawInfo* __restrict__ draw,
    int32_t* __restrict__ accepted_len, int32_t* __restrict__ next_tok) {
    __shared__ int s_rej[65];
    __shared__ int s_arg[65];
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    const int nch = n_chunks(V);
    const int row0 = cu_q[r];
    const int l = cu_q[r + 1] - row0 - 1;
    if (l < 0 || l > K || row0 < 0 || (int64_t)row0 + l + 1 > (int64_t)R * (K + 1)) {
        if (tid == 0) {
            accepted_len[r] = -1;
            next_tok[r] = -1;
            if (!GREEDY) draw[r] = DrawInfo{0, 0, 0, 0};
        }
        return;
    }
    const size_t esz = BF16 ? 2 : 4;
    for (int t = wave; t <= l; t += kAccThreads / DSPARK_WAVE) {
        const int64_t row = row0 + t;
        float A, B;
        int arg;
        row_stats<GREEDY>(stats + row * nch, nch, A, B, arg);
        if (lane == 0) {
            int rej = 0;
            if (GREEDY) {
                if (t < l) rej = draft_tok[(int64_t)r * K + t] != arg;
                s_arg[t] = arg;
            } else {
                rows[row] = RowInfo{A, B, r, t};
                if (t < l) {
                    const int x = draft_tok[(int64_t)r * K + t];
                    if (x < 0 || x >= V) {
                        rej = 1;
                    } else {
                        const void* rp = (const char*)logits + (size_t)row * (size_t)ld * esz;
                        const float y = load_logit<BF16>(rp, x) * scale2;
                        const float pt = exp2f(y - A) / B;
                        const float pd = draft_p[((int64_t)r * K + t) * V + x];
                        const float ratio = pd > 0.0f ? pt / pd : __builtin_huge_valf();
                        rej = !(u[(int64_t)r * (K + 1) + t] < ratio);
                    }
                }
            }
            s_rej[t] = rej;
        }
    }
    __syncthreads();
    if (tid == 0) {
        int acc = l;
        for (int t = 0; t < l; ++t)
            if (s_rej[t]) { acc = t; break; }
        accepted_len[r] = acc;
        if (GREEDY) next_tok[r] = s_arg[acc];
        else draw[r] = DrawInfo{acc < l ? 2 : 1, row0 + acc, acc, 0};
    }
}

// ---------------------------------------------------------------- residual masses

// mass of max(0, p_t - p_d) per (request, chunk) for requests that rejected
template <bool BF16, bool VEC, bool PDVEC>
__global__ __launch_bounds__(kAccThreads) void acc_resid(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld, int R, int K,
    int V, float scale2, const RowInfo* __restrict__ rows, const DrawInfo* __restrict__ draw,
    double* __restrict__ mass) {
    __shared__ double s_w[kAccThreads / DSPARK_WAVE];
    const int nch = n_chunks(V);
    const int64_t items = (int64_t)R * nch;
    const int lane = threadIdx.x & (DSPARK_WAVE - 1);
    const int wave = threadIdx.x / DSPARK_WAVE;
    const size_t esz = BF16 ? 2 : 4;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int r = (int)(it / nch);
        const int c = (int)(it - (int64_t)r * nch);
        const DrawInfo d = draw[r];
        if (d.kind != 2) continue;  // uniform across the block
        const RowInfo ri = rows[d.row];
        const int v0 = c * kChunk;
        const int v1 = min(V, v0 + kChunk);
        const void* rp = (const char*)logits + (size_t)d.row * (size_t)ld * esz;
        const float* pd = draft_p + ((int64_t)r * K + d.t) * V;
        float x[kPerThread], q[kPerThread];
        load_chunk<BF16, VEC>(rp, v0, v1, x);
        load_draft<BF16, VEC && PDVEC>(pd, v0, v1, q);
        const float invS = 1.0f / ri.S;
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            // positions past v1 have x = -inf: exp2 gives 0 and the term vanishes
            const float pt = exp2f(x[e] * scale2 - ri.M) * invS;
            acc += fmaxf(pt - q[e], 0.0f);
        }
        double w = wave_sum_f64((double)acc);
        if (lane == 0) s_w[wave] = w;
        __syncthreads();
        if (threadIdx.x == 0) {
            double t = 0.0;
            for (int q = 0; q < kAccThreads / DSPARK_WAVE; ++q) t += s_w[q];
            mass[(int64_t)r * nch + c] = t;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------- draw

template <bool BF16>
__global__ __launch_bounds__(kAccThreads) void acc_draw(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld,
    const float* __restrict__ u, int R, int K, int V, float scale2,
    const ChunkStat* __restrict__ stats, const RowInfo* __restrict__ rows,
    const DrawInfo* __restrict__ draw, const double* __restrict__ mass,
    int32_t* __restrict__ next_tok) {
    __shared__ double s_w[kMaxChunks];
    __shared__ int s_chunk;
    __shared__ double s_thr;
    __shared__ int s_kind;
    __shared__ double s_scan[kAccThreads / DSPARK_WAVE];
    __shared__ int s_pick;
    __shared__ int s_last;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    const int nch = n_chunks(V);
    const DrawInfo d = draw[r];
    if (d.kind == 0) return;
    const RowInfo ri = rows[d.row];
    const ChunkStat* st = stats + (int64_t)d.row * nch;
    const double uu = (double)u[(int64_t)r * (K + 1) + K];
    // chunk masses, in the units of the element masses used below
    int kind = d.kind;
    if (kind == 2) {
        double t = 0.0;
        for (int c = tid; c < nch; c += kAccThreads) t += mass[(int64_t)r * nch + c];
        t = wave_sum_f64(t);
        if (lane == 0) s_scan[wave] = t;
        __syncthreads();
        double tot = 0.0;
        for (int q = 0; q < kAccThreads / DSPARK_WAVE; ++q) tot += s_scan[q];
        if (!(tot > 0.0)) kind = 1;  // empty residual: draw from the target row
        __syncthreads();
    }
    for (int c = tid; c < nch; c += kAccThreads) {
        const ChunkStat x = st[c];
        s_w[c] = kind == 2 ? mass[(int64_t)r * nch + c]
                           : (x.a > -__builtin_huge_valf()
                                  ? (double)x.b * (double)exp2f(x.a - ri.M) : 0.0);
    }
    __syncthreads();
    if (tid == 0) {
        double tot = 0.0;
        for (int c = 0; c < nch; ++c) tot += s_w[c];
        const double thr = uu * tot;
        double cum = 0.0, before = 0.0;
        int pick = -1, lastpos = 0;
        for (int c = 0; c < nch; ++c) {
            const double w = s_w[c];
            if (w > 0.0) lastpos = c;
            if (pick < 0 && cum + w > thr) { pick = c; before = cum; }
            cum += w;
        }
        if (pick < 0) {  // rounding pushed u*total past the end: last non-empty chunk
            pick = lastpos;
            before = cum - s_w[pick];
        }
        s_chunk = pick;
        s_thr = thr - before;
        s_kind = kind;
        s_pick = 0x7fffffff;
        s_last = -1;
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
    const float invS = 1.0f / ri.S;
    // this thread's contiguous slice [first, first + kPerThread) of the chunk
    const int first = v0 + tid * kPerThread;
    float x[kPerThread], q[kPerThread];
    const bool full = first + kPerThread <= v1;
    const bool xvec = full && ((uintptr_t)rp % 16 == 0);
    if (xvec && BF16) {
        const u32x4* p4 = (const u32x4*)((const uint16_t*)rp + first);
#pragma unroll
        for (int k = 0; k < kPerThread / 8; ++k) {
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
        for (int k = 0; k < kPerThread / 4; ++k) {
            const f32x4 w = p4[k];
            x[4 * k] = w[0]; x[4 * k + 1] = w[1]; x[4 * k + 2] = w[2]; x[4 * k + 3] = w[3];
        }
    } else {
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const float xv = load_logit<BF16>(rp, min(first + e, v1 - 1));
            x[e] = first + e < v1 ? xv : -__builtin_huge_valf();
        }
    }
    if (kind == 2) {
        if (full && ((uintptr_t)(pd + first) % 16 == 0)) {
            const f32x4* p4 = (const f32x4*)(pd + first);
#pragma unroll
            for (int k = 0; k < kPerThread / 4; ++k) {
                const f32x4 w = p4[k];
                q[4 * k] = w[0]; q[4 * k + 1] = w[1]; q[4 * k + 2] = w[2]; q[4 * k + 3] = w[3];
            }
        } else {
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) {
                const float qv = pd[min(first + e, v1 - 1)];
                q[e] = first + e < v1 ? qv : 0.0f;
            }
        }
    }
    float wv[kPerThread];
    double loc = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const float y = x[e] * scale2;
        float m;
        if (kind == 2) m = fmaxf(exp2f(y - ri.M) * invS - q[e], 0.0f);
        else m = exp2f(y - ri.M);
        if (first + e >= v1) m = 0.0f;
        wv[e] = m;
        loc += (double)m;
        if (m > 0.0f) lastpos = first + e;
    }
    // exclusive scan of the per-thread sums over the block
    double incl = loc;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl += t;
    }
    if (lane == DSPARK_WAVE - 1) s_scan[wave] = incl;
    __syncthreads();
    double pre = incl - loc;
    for (int k = 0; k < wave; ++k) pre += s_scan[k];
    // the smallest index whose running mass exceeds thr; threads past the
    // crossing also propose a candidate, and the minimum wins
    if (pre + loc > thr) {
        double cum = pre;
        for (int e = 0; e < kPerThread; ++e) {
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

template <bool BF16, bool VEC, bool PDVEC>
__global__ __launch_bounds__(kAccThreads) void acc_rate_pass(
    const float* __restrict__ draft_p, const void* __restrict__ logits, int64_t ld,
    const int32_t* __restrict__ cu_q, int R, int K, int V, float scale2,
    const RowInfo* __restrict__ rows, double* __restrict__ part) {
    __shared__ double s_w[kAccThreads / DSPARK_WAVE];
    const int nch = n_chunks(V);
    const int64_t items = (int64_t)clamp_rows(cu_q[R], R * (K + 1)) * nch;
    const int lane = threadIdx.x & (DSPARK_WAVE - 1);
    const int wave = threadIdx.x / DSPARK_WAVE;
    const size_t esz = BF16 ? 2 : 4;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int64_t row = it / nch;
        const int c = (int)(it - row * nch);
        const RowInfo ri = rows[row];
        const int r = ri.req;
        // uniform across the block: rows of malformed requests and bonus rows carry no draft
        if (r < 0 || r >= R || ri.t < 0 || ri.t >= K) continue;
        const int ql = cu_q[r + 1] - cu_q[r];
        if (ri.t >= ql - 1) continue;
        const int v0 = c * kChunk;
        const int v1 = min(V, v0 + kChunk);
        const void* rp = (const char*)logits + (size_t)row * (size_t)ld * esz;
        const float* pd = draft_p + ((int64_t)r * K + ri.t) * V;
        float x[kPerThread], q[kPerThread];
        load_chunk<BF16, VEC>(rp, v0, v1, x);
        load_draft<BF16, VEC && PDVEC>(pd, v0, v1, q);
        const float invS = 1.0f / ri.S;
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e)
            acc += fminf(exp2f(x[e] * scale2 - ri.M) * invS, q[e]);
        double w = wave_sum_f64((double)acc);
        if (lane == 0) s_w[wave] = w;
        __syncthreads();
        if (threadIdx.x == 0) {
            double t = 0.0;
            for (int q = 0; q < kAccThreads / DSPARK_WAVE; ++q) t += s_w[q];
            part[row * nch + c] = t;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kAccThreads) void acc_rate_final(
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

template <bool BF16>
static hipError_t launch_typed(const AcceptArgs& a, void* ws, hipStream_t s) {
    const AccWs w = carve(ws, a.R, a.K, a.V);
    const int nch = n_chunks(a.V);
    const float scale2 = a.inv_temp * kLog2e;
    const bool greedy = a.draft_p == nullptr && a.u == nullptr;
    const size_t esz = BF16 ? 2 : 4;
    const bool vec = ((uintptr_t)a.logits % 16 == 0) && ((size_t)a.ld * esz) % 16 == 0;
    const int max_rows = a.R * (a.K + 1);
    const int64_t max_items = (int64_t)max_rows * nch;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(max_items, 2048));
    const dim3 blk(kAccThreads);
#define DS_ROWPASS(G, VV)                                                                    \
    hipLaunchKernelGGL((acc_rowpass<BF16, G, VV>), dim3(grid), blk, 0, s, a.logits, a.ld,  \
                       a.cu_q, a.R, a.V, max_rows, scale2, w.stats)
    if (greedy) { if (vec) DS_ROWPASS(true, true); else DS_ROWPASS(true, false); }
    else { if (vec) DS_ROWPASS(false, true); else DS_ROWPASS(false, false); }
#undef DS_ROWPASS
    hipError_t e = hipGetLastError();
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
    const int rgrid = (int)std::max<int64_t>(1, std::min<int64_t>((int64_t)a.R * nch, 2048));
    // draft rows start at multiples of V floats: 16-byte aligned when V % 4 == 0
    const bool pdvec = a.V % 4 == 0 && ((uintptr_t)a.draft_p % 16) == 0;
#define DS_RESID(VV, PV)                                                                      \
    hipLaunchKernelGGL((acc_resid<BF16, VV, PV>), dim3(rgrid), blk, 0, s, a.draft_p, a.logits, \
                       a.ld, a.R, a.K, a.V, scale2, w.rows, w.draw, w.mass)
    if (vec && pdvec) DS_RESID(true, true); else if (vec) DS_RESID(true, false); else DS_RESID(false, false);
#undef DS_RESID
    hipLaunchKernelGGL((acc_draw<BF16>), dim3(a.R), blk, 0, s, a.draft_p, a.logits, a.ld, a.u,
                       a.R, a.K, a.V, scale2, w.stats, w.rows, w.draw, w.mass, a.next_tok);
    if (a.accept_rate) {
#define DS_RATE(VV, PV)                                                                      \
        hipLaunchKernelGGL((acc_rate_pass<BF16, VV, PV>), dim3(grid), blk, 0, s, a.draft_p,   \
                           a.logits, a.ld, a.cu_q, a.R, a.K, a.V, scale2, w.rows, w.rate)
        if (vec && pdvec) DS_RATE(true, true); else if (vec) DS_RATE(true, false); else DS_RATE(false, false);
#undef DS_RATE
        const int fgrid = (int)std::max<int64_t>(
            1, std::min<int64_t>(((int64_t)a.R * (a.K + 1) + kAccThreads - 1) / kAccThreads, 1024));
        hipLaunchKernelGGL(acc_rate_final, dim3(fgrid), blk, 0, s, a.cu_q, a.R, a.V, max_rows, w.rows,
                           w.rate, a.accept_rate);
    }
    return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, void* ws, hipStream_t s) {
    return a.logit_bf16 ? launch_typed<true>(a, ws, s) : launch_typed<false>(a, ws, s);
}

}  // namespace dspark
