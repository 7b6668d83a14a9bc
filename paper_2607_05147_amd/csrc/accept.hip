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

// Loads this thread's kPerThread consecutive logits of [v0, v1) into x[]
// (positions past v1 get -inf).  Vector path: 16-byte loads.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load_chunk(const void* row, int v0, int v1, float* x) {
    const int first = v0 + threadIdx.x * kPerThread;
    if (VEC && first + kPerThread <= v1) {
        if (BF16) {
            const u32x4* p = (const u32x4*)((const uint16_t*)row + first);
#pragma unroll
            for (int q = 0; q < kPerThread / 8; ++q) {
                const u32x4 w = __builtin_nontemporal_load(p + q);
                const uint32_t ww[4] = {w[0], w[1], w[2], w[3]};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[q * 8 + 2 * e] = __uint_as_float(ww[e] << 16);
                    x[q * 8 + 2 * e + 1] = __uint_as_float(ww[e] & 0xffff0000u);
                }
            }
        } else {
            const f32x4* p = (const f32x4*)((const float*)row + first);
#pragma unroll
            for (int q = 0; q < kPerThread / 4; ++q) {
                const f32x4 w = __builtin_nontemporal_load(p + q);
                x[q * 4 + 0] = w[0]; x[q * 4 + 1] = w[1]; x[q * 4 + 2] = w[2]; x[q * 4 + 3] = w[3];
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const int v = first + e;
            x[e] = v < v1 ? load_logit<BF16>(row, v) : -__builtin_huge_valf();
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
        const int first = v0 + threadIdx.x * kPerThread;
        if (GREEDY) {
            // thread-local max/argmax; the thread's first in-range element seeds it
            float best = x[0];
            int arg = first < v1 ? first : 0x7fffffff;
#pragma unroll
            for (int e = 1; e < kPerThread; ++e)
                if (x[e] > best) { best = x[e]; arg = first + e; }
            if (first >= v1) best = -__builtin_huge_valf();
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

template <bool BF16, bool GREEDY>
__global__ __launch_bounds__(kAccThreads) void acc_resolve(
    const int32_t* __restrict__ draft_tok, const float* __restrict__ draft_p,
    const void* __restrict__ logits, int64_t ld, const float* __restrict__ u,
    const int32_t* __restrict__ cu_q, int R, int K, int V, float scale2,
    const ChunkStat* __restrict__ stats, RowInfo* __restrict__ rows, DrawInfo* __restrict__ draw,
    int32_t* __restrict__ accepted_len, int32_t* __restrict__ next_tok) {
    __shared__ int s_rej[65];
    __shared__ int s_arg[65];
    __shared__ float s_M[65];
    __shared__ float s_S[65];
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
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
    if (tid <= l) {
        const int64_t row = row0 + tid;
        const ChunkStat* st = stats + row * nch;
        int rej = 0;
        if (GREEDY) {
            float best = st[0].a;
            int arg = st[0].arg;
            for (int c = 1; c < nch; ++c)
                if (st[c].a > best) { best = st[c].a; arg = st[c].arg; }
            if (tid < l) rej = draft_tok[(int64_t)r * K + tid] != arg;
            s_arg[tid] = arg;
        } else {
            float M = st[0].a;
            for (int c = 1; c < nch; ++c) M = fmaxf(M, st[c].a);
            float S = 0.0f;
            for (int c = 0; c < nch; ++c)
                if (st[c].a > -__builtin_huge_valf()) S += st[c].b * exp2f(st[c].a - M);
            rows[row] = RowInfo{M, S, r, tid};
            if (tid < l) {
                const int x = draft_tok[(int64_t)r * K + tid];
                if (x < 0 || x >= V) {
                    rej = 1;
                } else {
                    const void* rp = (const char*)logits + (size_t)row * (size_t)ld * esz;
                    const float y = load_logit<BF16>(rp, x) * scale2;
                    const float pt = exp2f(y - M) / S;
                    const float pd = draft_p[((int64_t)r * K + tid) * V + x];
                    const float ratio = pd > 0.0f ? pt / pd : __builtin_huge_valf();
                    rej = !(u[(int64_t)r * (K + 1) + tid] < ratio);
                }
            }
            s_M[tid] = M;
            s_S[tid] = S;
        }
        s_rej[tid] = rej;
    }
    __syncthreads();
    if (tid == 0) {
        int acc = l;
        for (int t = 0; t < l; ++t)
            if (s_rej[t]) { acc = t; break; }
        accepted_len[r] = acc;
        if (GREEDY) {
            next_tok[r] = s_arg[acc];
        } else {
            draw[r] = DrawInfo{acc < l ? 2 : 1, row0 + acc, acc, 0};
        }
    }
}

// ---------------------------------------------------------------- residual masses

// mass of max(0, p_t - p_d) per (request, chunk) for requests that rejected
template <bool BF16, bool VEC>
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
        float x[kPerThread];
        load_chunk<BF16, VEC>(rp, v0, v1, x);
        const int first = v0 + threadIdx.x * kPerThread;
        const float invS = 1.0f / ri.S;
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const int v = first + e;
            if (v < v1) {
                const float pt = exp2f(x[e] * scale2 - ri.M) * invS;
                acc += fmaxf(pt - pd[v], 0.0f);
            }
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
    if (tid == 0) {
        int kind = d.kind;
        if (kind == 2) {
            double tot = 0.0;
            for (int c = 0; c < nch; ++c) tot += mass[(int64_t)r * nch + c];
            if (!(tot > 0.0)) kind = 1;  // empty residual: draw from the target row
        }
        // chunk masses in the units of the element masses used below
        double tot = 0.0;
        for (int c = 0; c < nch; ++c) {
            const double w = kind == 2 ? mass[(int64_t)r * nch + c]
                                       : (st[c].a > -__builtin_huge_valf()
                                              ? (double)st[c].b * (double)exp2f(st[c].a - ri.M)
                                              : 0.0);
            tot += w;
        }
        const double thr = uu * tot;
        double cum = 0.0;
        int pick = -1, lastpos = 0;
        double before = 0.0;
        for (int c = 0; c < nch; ++c) {
            const double w = kind == 2 ? mass[(int64_t)r * nch + c]
                                       : (st[c].a > -__builtin_huge_valf()
                                              ? (double)st[c].b * (double)exp2f(st[c].a - ri.M)
                                              : 0.0);
            if (w > 0.0) lastpos = c;
            if (pick < 0 && cum + w > thr) { pick = c; before = cum; }
            cum += w;
        }
        if (pick < 0) {  // rounding pushed u*total past the end: take the last non-empty chunk
            pick = lastpos;
            before = cum - (kind == 2 ? mass[(int64_t)r * nch + pick]
                                      : (double)st[pick].b * (double)exp2f(st[pick].a - ri.M));
        }
        s_chunk = pick;
        s_thr = thr - before;
        s_kind = kind;
        s_pick = 0x7fffffff;
        s_last = -1;
    }
    __syncthreads();
    const int c = s_chunk;
    const int kind = s_kind;
    const double thr = s_thr;
    const int v0 = c * kChunk;
    const int v1 = min(V, v0 + kChunk);
    const size_t esz = BF16 ? 2 : 4;
    const void* rp = (const char*)logits + (size_t)d.row * (size_t)ld * esz;
    const float* pd = draft_p + ((int64_t)r * K + d.t) * V;
    const float invS = 1.0f / ri.S;
    const int first = v0 + tid * kPerThread;
    float w[kPerThread];
    double loc = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const int v = first + e;
        float m = 0.0f;
        if (v < v1) {
            const float y = load_logit<BF16>(rp, v) * scale2;
            if (kind == 2) {
                const float pt = exp2f(y - ri.M) * invS;
                m = fmaxf(pt - pd[v], 0.0f);
            } else {
                m = exp2f(y - ri.M);
            }
        }
        w[e] = m;
        loc += (double)m;
        if (m > 0.0f) lastpos = v;
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
    for (int q = 0; q < wave; ++q) pre += s_scan[q];
    // the smallest index whose running mass exceeds thr; threads past the
    // crossing also propose a candidate, and the minimum wins
    if (pre + loc > thr) {
        double cum = pre;
        for (int e = 0; e < kPerThread; ++e) {
            cum += (double)w[e];
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

template <bool BF16, bool VEC>
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
        float x[kPerThread];
        load_chunk<BF16, VEC>(rp, v0, v1, x);
        const int first = v0 + threadIdx.x * kPerThread;
        const float invS = 1.0f / ri.S;
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            const int v = first + e;
            if (v < v1) acc += fminf(exp2f(x[e] * scale2 - ri.M) * invS, pd[v]);
        }
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
    if (vec)
        hipLaunchKernelGGL((acc_resid<BF16, true>), dim3(rgrid), blk, 0, s, a.draft_p, a.logits,
                           a.ld, a.R, a.K, a.V, scale2, w.rows, w.draw, w.mass);
    else
        hipLaunchKernelGGL((acc_resid<BF16, false>), dim3(rgrid), blk, 0, s, a.draft_p,
                           a.logits, a.ld, a.R, a.K, a.V, scale2, w.rows, w.draw, w.mass);
    hipLaunchKernelGGL((acc_draw<BF16>), dim3(a.R), blk, 0, s, a.draft_p, a.logits, a.ld, a.u,
                       a.R, a.K, a.V, scale2, w.stats, w.rows, w.draw, w.mass, a.next_tok);
    if (a.accept_rate) {
        if (vec)
            hipLaunchKernelGGL((acc_rate_pass<BF16, true>), dim3(grid), blk, 0, s, a.draft_p,
                               a.logits, a.ld, a.cu_q, a.R, a.K, a.V, scale2, w.rows, w.rate);
        else
            hipLaunchKernelGGL((acc_rate_pass<BF16, false>), dim3(grid), blk, 0, s, a.draft_p,
                               a.logits, a.ld, a.cu_q, a.R, a.K, a.V, scale2, w.rows, w.rate);
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
