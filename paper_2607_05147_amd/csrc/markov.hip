// Markov-head draft block on gfx950: the drafter's sequential stage.
//
// For every request r, with x_0 = anchor[r] and k = 1 .. K (the left-to-right
// factorisation of the semi-autoregressive stage, eq. sequential-factorization,
// with the Markov head's low-rank transition bias of eq. markov, and the
// confidence head of eq. confidence with the per-position temperatures of its
// post-hoc calibration):
//   e_k = W1[x_{k-1}];   z_k = inv_temp * (U_k + W2^T e_k);   p_k = softmax(z_k);
//   x_k = inverse CDF of p_k at u[r, k-1];   c_k = sigmoid(w . [h_k; e_k] / T_k).
// Launches, all on one stream: md_hidden (the backbone part w_h . h_k of every
// confidence logit, once) and md_first (e_1 and c_1), then per position k:
//   md_tile<0>  one workgroup per 128 vocabulary entries: W2^T e for every
//               request on v_mfma_f32_16x16x32_bf16 (the tile's W2t rows stay
//               in registers as A operands, the embeddings stream through LDS
//               in chunks of 64 requests as B operands), plus the base logits;
//               then the tile's softmax statistics (max, sum of exp) per request;
//   md_stats    one wave per request: the row's max and total and the tile in
//               which the running mass passes u * total (fp64 prefix over the
//               tiles in vocabulary order);
//   md_tile<1>  the same product again, writing p_k = exp(z - max) / total; the
//               workgroup whose tile holds a request's draw makes it (fp64
//               prefix of that tile's masses), writes x_k, gathers e_{k+1} into
//               the other embedding buffer and writes c_{k+1}.
// The product is recomputed rather than stored: the second pass reads W2t
// again (66 MB at V = 129280, rank 256, which the 256 MB last-level cache can
// hold) instead of writing and re-reading fp32 logits.  The positions of a
// block are sequential by definition (x_k feeds position k + 1).
#include <algorithm>
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace dspark {
namespace mkd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / DSPARK_WAVE;
constexpr int kTileV = 128;              // vocabulary entries per workgroup tile
constexpr int kWaveV = kTileV / kWaves;  // 32 per wave
constexpr int kVT = kWaveV / 16;         // 16-entry blocks per wave
constexpr int kChunkR = 32;              // requests per LDS chunk
constexpr int kRT = kChunkR / 16;        // 16-request blocks per chunk

__host__ __device__ constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Slot of 16-byte chunk c in row t of the embedding chunk (nch chunks per row,
// a power of two).  The XOR (bits of t in the order 0, 2, 1, 3) puts the 16
// lanes of every phase of the B-operand reads on distinct banks for every
// supported rank (gfx950 serves a 16-byte LDS read in four 16-lane phases split
// by lane bit 5 and the parity of lane bits 2 ^ 3 ^ 4).
__device__ __forceinline__ int eslot(int t, int c, int nch) {
    const int f = (t & 1) | (((t >> 2) & 1) << 1) | (((t >> 1) & 1) << 2) | (((t >> 3) & 1) << 3);
    return c ^ (f & (nch - 1));
}

__device__ __forceinline__ float block_sum(float v, float* s) {
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) s[wave] = v;
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += s[w];
    return t;
}

__device__ __forceinline__ float block_max(float v, float* s) {
    v = wave_max(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) s[wave] = v;
    __syncthreads();
    float t = -__builtin_huge_valf();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t = fmaxf(t, s[w]);
    return t;
}

// Inclusive prefix sum over the block in thread order (fp64); *total gets the sum.
__device__ __forceinline__ double block_scan(double v, double* s, double* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    double incl = v;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl += t;
    }
    __syncthreads();
    if (lane == DSPARK_WAVE - 1) s[wave] = incl;
    __syncthreads();
    double before = 0.0, all = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        if (w < wave) before += s[w];
        all += s[w];
    }
    *total = all;
    return before + incl;
}

__device__ __forceinline__ float load_base(const MarkovArgs& a, int64_t i) {
    return a.base_bf16 ? bf16_to_f32(((const uint16_t*)a.base)[i]) : ((const float*)a.base)[i];
}

// token of position k - 1 (the anchor for k = 1); -1 when it is not a valid token
__device__ __forceinline__ int prev_token(const MarkovArgs& a, int r, int k) {
    const int x = k == 1 ? a.anchor[r] : a.draft_tok[(int64_t)r * a.K + (k - 2)];
    return x >= 0 && x < a.V ? x : -1;
}

// Maximum / sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the lanes that
// hold one request's entries of a block), with lane swaps instead of LDS.
__device__ __forceinline__ float quad_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Per-request state of a position between the two tile passes.
struct RowInfo {
    float M;     // row maximum of z (base-2 units: z * log2 e)
    float S;     // sum over the row of exp(z - M)
    int tile;    // tile in which the running mass passes u * S
    int pad;
    double thr;  // u * S minus the mass of the tiles before `tile` (+inf: the tile's last entry with mass)
};

// w_e . W1[x] over one wave (every lane gets the sum)
__device__ __forceinline__ float embed_dot(const MarkovArgs& a, const uint16_t* w1, int lane) {
    float s = 0.0f;
    for (int j = lane; j < a.rank; j += DSPARK_WAVE) s += a.w_conf[a.d + j] * bf16_to_f32(w1[j]);
    return wave_sum(s);
}

__device__ __forceinline__ float confidence(const MarkovArgs& a, float logit, int k) {
    const float T = a.sts_temp ? a.sts_temp[k - 1] : 1.0f;
    return 1.0f / (1.0f + expf(-logit / T));
}

// --------------------------------------------------------------- md_hidden

// The backbone part of every confidence logit, w_h . h_k, for all (r, k):
// one wave per row (independent of the drawn tokens, so done once up front).
__global__ __launch_bounds__(kThreads) void md_hidden(MarkovArgs a, float* sh) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * kWaves + wave;
    if (row >= (int64_t)a.R * a.K) return;  // whole wave
    const uint16_t* h = a.hidden + row * a.d;
    float s = 0.0f;
    if ((a.d & 7) == 0 && ((uintptr_t)a.hidden & 15) == 0) {
        for (int i = lane * 8; i < a.d; i += DSPARK_WAVE * 8) {
            const uint4 hv = *(const uint4*)(h + i);
            const uint32_t w4[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
            for (int q = 0; q < 4; ++q)
                s += a.w_conf[i + 2 * q] * __uint_as_float(w4[q] << 16) +
                     a.w_conf[i + 2 * q + 1] * __uint_as_float(w4[q] & 0xffff0000u);
        }
    } else {
        for (int i = lane; i < a.d; i += DSPARK_WAVE) s += a.w_conf[i] * bf16_to_f32(h[i]);
    }
    s = wave_sum(s);
    if (lane == 0) sh[row] = s;
}

// ---------------------------------------------------------------- md_first

// Position 1: e_1 = W1[x_0] into the first embedding buffer, and c_1.  One wave per request.
__global__ __launch_bounds__(kThreads) void md_first(MarkovArgs a, const float* sh, uint16_t* E0) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int r = blockIdx.x * kWaves + wave;
    if (r >= a.R) return;  // whole wave
    const int x0 = a.anchor[r];
    const bool ok = x0 >= 0 && x0 < a.V;
    const uint16_t* w1 = a.W1 + (int64_t)(ok ? x0 : 0) * a.rank;
    for (int j = lane * 8; j < a.rank; j += DSPARK_WAVE * 8)
        *(uint4*)(E0 + (int64_t)r * a.rank + j) = *(const uint4*)(w1 + j);
    const float s = embed_dot(a, w1, lane) + (sh ? sh[(int64_t)r * a.K] : 0.0f);
    if (lane == 0) a.conf[(int64_t)r * a.K] = ok ? confidence(a, s, 1) : __builtin_nanf("");
}

// ----------------------------------------------------------------- md_tile

// z for (request, vocabulary entry) pairs of one 128-entry tile:
// C[v, r] = sum_j W2t[v, j] E[r, j] on MFMA (A: the tile's W2t rows, kept in
// registers; B: the embeddings, 64 requests at a time through LDS), then
// z = inv_temp * (U + C), kept in base-2 units (z * log2 e, so that exp(z - m)
// is one v_exp_f32 of the difference).
// PASS 0: per-tile statistics stats[r * ntiles + tile] = (max z, sum 2^(z - max)).
// PASS 1: draft_p = 2^(z - M) / S with (M, S) of the request's RowInfo; for
//   every request whose draw falls in this tile, the draw itself (fp64 prefix
//   of the tile's masses in vocabulary order), and for position k < K the next
//   embedding E_next[r] = W1[x_k] and the confidence c_{k+1}.
// VEC: 4 consecutive entries per lane are loaded / stored as one vector
// (V, ld multiples of 4, aligned rows).
template <int KS, int PASS, bool VEC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 4))) void md_tile(MarkovArgs a, const uint16_t* E,
                                                    float2* stats, const RowInfo* info,
                                                    uint16_t* E_next, const float* sh,
                                                    int ntiles, int k) {
    constexpr int kNch = 4 * KS;  // 16-byte chunks per embedding row
    constexpr int kRank = 32 * KS;
    __shared__ __align__(16) uint16_t se[kChunkR * kRank];
    __shared__ float2 sst[kWaves][kChunkR];
    __shared__ float smass[kTileV];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const int tile = blockIdx.x;
    const int v0 = tile * kTileV + wave * kWaveV;
    constexpr float kLog2e = 1.4426950408889634f;
    const float scale2 = a.inv_temp * kLog2e;

    // A fragments: W2t rows v0 + 16 vt + lr (clamped into the vocabulary), dims 32 ks + 8 lq ..
    bf16x8 af[kVT][KS];
#pragma unroll
    for (int vt = 0; vt < kVT; ++vt) {
        const int v = min(v0 + 16 * vt + lr, a.V - 1);
        const uint16_t* src = a.W2t + (int64_t)v * kRank + 8 * lq;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) af[vt][ks] = *(const bf16x8*)(src + 32 * ks);
    }

    for (int c0 = 0; c0 < a.R; c0 += kChunkR) {
        const bool interior = (tile + 1) * kTileV <= a.V && c0 + kChunkR <= a.R;
        // the chunk's embeddings first, then its base logits: the LDS stores
        // below wait only for the embeddings (loads complete in order), and the
        // base logits stay in flight during the products
        constexpr int kCopy = ceil_div(kChunkR * kNch, kThreads);
        uint4 ev[kCopy];
#pragma unroll
        for (int i = 0; i < kCopy; ++i) {
            const int idx = tid + i * kThreads;
            const int t = idx / kNch, c = idx - t * kNch;
            ev[i] = idx < kChunkR * kNch && c0 + t < a.R ? *(const uint4*)(E + (int64_t)(c0 + t) * kRank + 8 * c)
                                                          : uint4{0u, 0u, 0u, 0u};
        }
        float ub[kRT][kVT][4];
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int r = min(c0 + 16 * rt + lr, a.R - 1);
            const int64_t row = (int64_t)r * a.K + (k - 1);
#pragma unroll
            for (int vt = 0; vt < kVT; ++vt) {
                const int vb = v0 + 16 * vt + 4 * lq;
                if (VEC && vb + 3 < a.V) {
                    if (a.base_bf16) {
                        const uint2 w = *(const uint2*)((const uint16_t*)a.base + row * a.ld + vb);
                        ub[rt][vt][0] = __uint_as_float(w.x << 16);
                        ub[rt][vt][1] = __uint_as_float(w.x & 0xffff0000u);
                        ub[rt][vt][2] = __uint_as_float(w.y << 16);
                        ub[rt][vt][3] = __uint_as_float(w.y & 0xffff0000u);
                    } else {
                        const float4 w = *(const float4*)((const float*)a.base + row * a.ld + vb);
                        ub[rt][vt][0] = w.x, ub[rt][vt][1] = w.y, ub[rt][vt][2] = w.z, ub[rt][vt][3] = w.w;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        ub[rt][vt][e] = vb + e < a.V ? load_base(a, row * a.ld + vb + e) : 0.0f;
                }
            }
        }
        lds_barrier();  // the previous chunk's LDS reads are done (global loads stay in flight)
#pragma unroll
        for (int i = 0; i < kCopy; ++i) {
            const int idx = tid + i * kThreads;
            const int t = idx / kNch, c = idx - t * kNch;
            if (idx < kChunkR * kNch) *(uint4*)(se + (t * kNch + eslot(t, c, kNch)) * 8) = ev[i];
        }
        lds_barrier();

        // lane holds C[v, r] for v = v0 + 16 vt + 4 lq + e, r = c0 + 16 rt + lr
        f32x4 acc[kVT][kRT];
#pragma unroll
        for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) acc[vt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int t = 16 * rt + lr;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 b = *(const bf16x8*)(se + (t * kNch + eslot(t, 4 * ks + lq, kNch)) * 8);
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
                    acc[vt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[vt][ks], b, acc[vt][rt], 0, 0, 0);
            }
        }

#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int r = c0 + 16 * rt + lr;
            const bool rok = r < a.R;
            float z[kVT][4];
#pragma unroll
            for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                for (int e = 0; e < 4; ++e) z[vt][e] = scale2 * (ub[rt][vt][e] + acc[vt][rt][e]);
            if (!interior) {  // the vocabulary's last tile or the requests' last chunk
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (!(rok && v0 + 16 * vt + 4 * lq + e < a.V)) z[vt][e] = -__builtin_huge_valf();
            }
            if (PASS == 0) {
                float m = -__builtin_huge_valf();
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) m = fmaxf(m, z[vt][e]);
                m = quad_max(m);
                float s = 0.0f;
                if (m > -__builtin_huge_valf()) {
#pragma unroll
                    for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                        for (int e = 0; e < 4; ++e) s += __builtin_amdgcn_exp2f(z[vt][e] - m);
                }
                s = quad_sum(s);
                if (lq == 0) sst[wave][16 * rt + lr] = float2{m, s};
            } else {
                const RowInfo ri = info[rok ? r : 0];
                const float inv = 1.0f / ri.S;
                float q[kVT][4];
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) q[vt][e] = __builtin_amdgcn_exp2f(z[vt][e] - ri.M);
                if (rok) {
                    float* out = a.draft_p + ((int64_t)r * a.K + (k - 1)) * a.V;
#pragma unroll
                    for (int vt = 0; vt < kVT; ++vt) {
                        const int vb = v0 + 16 * vt + 4 * lq;
                        if (VEC && vb + 3 < a.V) {
                            *(float4*)(out + vb) = float4{q[vt][0] * inv, q[vt][1] * inv, q[vt][2] * inv,
                                                          q[vt][3] * inv};
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (vb + e < a.V) out[vb + e] = q[vt][e] * inv;
                        }
                    }
                }
                // draws that fall in this tile (the same set in every wave)
                uint64_t bits = __builtin_amdgcn_ballot_w64(rok && lq == 0 && ri.tile == tile);
                while (bits) {
                    const int j = __builtin_ctzll(bits);
                    bits &= bits - 1;
                    if (lr == j) {
#pragma unroll
                        for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                            for (int e = 0; e < 4; ++e) smass[wave * kWaveV + 16 * vt + 4 * lq + e] = q[vt][e];
                    }
                    lds_barrier();
                    if (wave == 0) {
                        const int rr = c0 + 16 * rt + j;
                        const int64_t row = (int64_t)rr * a.K + (k - 1);
                        const double thr = info[rr].thr;
                        const double m0 = smass[2 * lane], m1 = smass[2 * lane + 1];
                        double incl = m0 + m1;
#pragma unroll
                        for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
                            const double t = __shfl_up(incl, o, DSPARK_WAVE);
                            if (lane >= o) incl += t;
                        }
                        const double c0m = incl - (m0 + m1);  // mass before entry 2 * lane
                        // first entry whose running mass passes thr (zero masses are never drawn)
                        const int cand = c0m + m0 > thr && m0 > 0.0 ? 2 * lane
                                         : incl > thr && m1 > 0.0   ? 2 * lane + 1
                                                                    : kTileV;
                        int first = cand;
#pragma unroll
                        for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o, DSPARK_WAVE));
                        // rounding: the tile's last entry with mass
                        int last = m1 > 0.0 ? 2 * lane + 1 : m0 > 0.0 ? 2 * lane : -1;
#pragma unroll
                        for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, DSPARK_WAVE));
                        const int pick = first < kTileV ? first : max(last, 0);
                        const int x = tile * kTileV + pick;
                        const bool ok = prev_token(a, rr, k) >= 0;
                        if (lane == 0) a.draft_tok[row] = ok ? x : -1;
                        if (k < a.K) {
                            const uint16_t* w1 = a.W1 + (int64_t)(ok ? x : 0) * a.rank;
                            for (int q8 = lane * 8; q8 < a.rank; q8 += DSPARK_WAVE * 8)
                                *(uint4*)(E_next + (int64_t)rr * a.rank + q8) = *(const uint4*)(w1 + q8);
                            const float sc = embed_dot(a, w1, lane) + (sh ? sh[row + 1] : 0.0f);
                            if (lane == 0) a.conf[row + 1] = ok ? confidence(a, sc, k + 1) : __builtin_nanf("");
                        }
                    }
                    lds_barrier();
                }
            }
        }
        if (PASS == 0) {
            lds_barrier();
            if (tid < kChunkR && c0 + tid < a.R) {
                float M = -__builtin_huge_valf();
#pragma unroll
                for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sst[w][tid].x);
                float S = 0.0f;
                if (M > -__builtin_huge_valf()) {
#pragma unroll
                    for (int w = 0; w < kWaves; ++w)
                        if (sst[w][tid].x > -__builtin_huge_valf()) S += sst[w][tid].y * exp2f(sst[w][tid].x - M);
                }
                stats[(int64_t)(c0 + tid) * ntiles + tile] = float2{M, S};
            }
        }
    }
}

// ---------------------------------------------------------------- md_stats

// Per request (one workgroup): the row maximum and total from the tile
// statistics (tile masses in fp64), and the tile in which the running mass
// passes u * total, scanning the tiles in vocabulary order.
constexpr int kStatsPer = 8;  // tiles per thread (up to 2048 tiles: V <= 262144)
__global__ __launch_bounds__(kThreads) void md_stats(MarkovArgs a, const float2* stats, RowInfo* info,
                                                     int ntiles, int k) {
    __shared__ float s_f[kWaves];
    __shared__ double s_d[kWaves];
    __shared__ int s_pick, s_last;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const float2* st = stats + (int64_t)r * ntiles;
    const int per = ceil_div(ntiles, kThreads);  // a contiguous run of tiles per thread
    const int t0 = tid * per;
    float2 x[kStatsPer];
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int i = 0; i < kStatsPer; ++i) {
        x[i] = i < per && t0 + i < ntiles ? st[t0 + i] : float2{-__builtin_huge_valf(), 0.0f};
        m = fmaxf(m, x[i].x);
    }
    const float M = block_max(m, s_f);
    double w[kStatsPer], loc = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int i = 0; i < kStatsPer; ++i) {
        w[i] = x[i].x > -__builtin_huge_valf() ? (double)x[i].y * (double)exp2f(x[i].x - M) : 0.0;
        loc += w[i];
        if (w[i] > 0.0) lastpos = t0 + i;
    }
    double total;
    const double incl = block_scan(loc, s_d, &total);
    const double thr = (double)a.u[(int64_t)r * a.K + (k - 1)] * total;
    if (tid == 0) {
        s_pick = kThreads;
        s_last = -1;
    }
    __syncthreads();
    if (incl > thr && loc > 0.0) atomicMin(&s_pick, tid);
    if (lastpos >= 0) atomicMax(&s_last, lastpos);
    __syncthreads();
    RowInfo ri;
    ri.M = M;
    ri.S = (float)total;
    ri.pad = 0;
    if (tid == s_pick) {
        double cum = incl - loc;
        int pick = -1;
        double before = 0.0;
#pragma unroll
        for (int i = 0; i < kStatsPer; ++i) {
            if (pick < 0 && w[i] > 0.0 && cum + w[i] > thr) {
                pick = t0 + i;
                before = cum;
            }
            cum += w[i];
        }
        if (pick >= 0) {
            ri.tile = pick;
            ri.thr = thr - before;
        } else {  // rounding inside the run: its last tile with mass
            ri.tile = lastpos;
            ri.thr = __builtin_huge_val();
        }
        info[r] = ri;
    } else if (s_pick == kThreads && tid == 0) {
        // rounding pushed u * total past the end: the row's last tile with mass
        ri.tile = max(s_last, 0);
        ri.thr = __builtin_huge_val();
        info[r] = ri;
    }
}

template <int KS>
hipError_t launch_ks(const MarkovArgs& a, uint16_t* E0, uint16_t* E1, float2* stats, RowInfo* info,
                     float* sh, int ntiles, bool vec, hipStream_t s) {
    const int64_t rows = (int64_t)a.R * a.K;
    if (a.d > 0) hipLaunchKernelGGL(md_hidden, dim3((unsigned)ceil_div((int)rows, kWaves)), dim3(kThreads), 0, s, a, sh);
    const float* shp = a.d > 0 ? sh : nullptr;
    hipLaunchKernelGGL(md_first, dim3(ceil_div(a.R, kWaves)), dim3(kThreads), 0, s, a, shp, E0);
    for (int k = 1; k <= a.K; ++k) {
        uint16_t* Ek = (k & 1) ? E0 : E1;
        uint16_t* En = (k & 1) ? E1 : E0;
        if (vec) hipLaunchKernelGGL((md_tile<KS, 0, true>), dim3(ntiles), dim3(kThreads), 0, s, a, Ek, stats, info, En, shp, ntiles, k);
        else hipLaunchKernelGGL((md_tile<KS, 0, false>), dim3(ntiles), dim3(kThreads), 0, s, a, Ek, stats, info, En, shp, ntiles, k);
        hipLaunchKernelGGL(md_stats, dim3(a.R), dim3(kThreads), 0, s, a, stats, info, ntiles, k);
        if (vec) hipLaunchKernelGGL((md_tile<KS, 1, true>), dim3(ntiles), dim3(kThreads), 0, s, a, Ek, stats, info, En, shp, ntiles, k);
        else hipLaunchKernelGGL((md_tile<KS, 1, false>), dim3(ntiles), dim3(kThreads), 0, s, a, Ek, stats, info, En, shp, ntiles, k);
    }
    return hipGetLastError();
}

}  // namespace mkd

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

namespace {
struct WsLayout {
    size_t e, stats, info, sh, total;
};
WsLayout ws_layout(int R, int K, int V, int rank) {
    const int ntiles = mkd::ceil_div(V, mkd::kTileV);
    WsLayout l;
    l.e = align256((size_t)R * rank * 2);
    l.stats = align256((size_t)R * ntiles * sizeof(float2));
    l.info = align256((size_t)R * sizeof(mkd::RowInfo));
    l.sh = align256((size_t)R * K * sizeof(float));
    l.total = 2 * l.e + l.stats + l.info + l.sh;
    return l;
}
}  // namespace

size_t markov_workspace(int R, int K, int V, int rank) { return ws_layout(R, K, V, rank).total; }

bool markov_rank_supported(int rank) { return rank == 32 || rank == 64 || rank == 128 || rank == 256; }

int markov_max_vocab() { return mkd::kThreads * mkd::kStatsPer * mkd::kTileV; }

hipError_t launch_markov(const MarkovArgs& a, void* ws, hipStream_t s) {
    const int ntiles = mkd::ceil_div(a.V, mkd::kTileV);
    const WsLayout l = ws_layout(a.R, a.K, a.V, a.rank);
    char* p = (char*)ws;
    uint16_t* E0 = (uint16_t*)p;
    uint16_t* E1 = (uint16_t*)(p + l.e);
    float2* stats = (float2*)(p + 2 * l.e);
    mkd::RowInfo* info = (mkd::RowInfo*)(p + 2 * l.e + l.stats);
    float* sh = (float*)(p + 2 * l.e + l.stats + l.info);
    const size_t eb = a.base_bf16 ? 2 : 4;
    const bool vec = a.V % 4 == 0 && a.ld % 4 == 0 && ((uintptr_t)a.base % (4 * eb)) == 0 &&
                     ((uintptr_t)a.draft_p % 16) == 0;
    switch (a.rank) {
        case 32: return mkd::launch_ks<1>(a, E0, E1, stats, info, sh, ntiles, vec, s);
        case 64: return mkd::launch_ks<2>(a, E0, E1, stats, info, sh, ntiles, vec, s);
        case 128: return mkd::launch_ks<4>(a, E0, E1, stats, info, sh, ntiles, vec, s);
        default: return mkd::launch_ks<8>(a, E0, E1, stats, info, sh, ntiles, vec, s);
    }
}

}  // namespace dspark
